"""fp64 CPU oracle for paged grouped-query decode attention.

TEST INFRASTRUCTURE ONLY.  Only the test-suite, the smoke check and the
benchmark's CPU-baseline leg may import this package.  It shares no code with
the GPU library and imports nothing from it.

The arithmetic lives in ``decode_attn_oracle.c`` (plain C, fp64); this module
only compiles it with gcc and marshals numpy arrays through ctypes.  The
operation is the scaled dot-product attention of one decode step over a paged
KV cache (the paper's rollout phase, Sec. 2.1; its paged KV cache, Sec. 1):
``out[b,h] = softmax(scale * q[b,h] . K_b^T) V_b`` with ``K_b``/``V_b`` the
first ``seq_lens[b]`` cached tokens of sequence ``b``, gathered through the
block table, and KV head ``h // (Hq // Hkv)``.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "decode_attn_oracle.c")
LIB_PATH = os.path.join(_HERE, "libdecode_attn_oracle.so")

KV_BF16 = 0
KV_FP8_E4M3 = 1

LAYOUT_HND = 0   # pools [page][kv head][slot][dim]
LAYOUT_NHD = 1   # pools [page][slot][kv head][dim]

OK = 0
ERR_ARG = 1
ERR_PRECONDITION = 2
ERR_NOMEM = 3


class OracleError(RuntimeError):
    pass


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (-O2, OpenMP, no FMA contraction)."""
    if not force and os.path.exists(LIB_PATH):
        return LIB_PATH
    tmp = LIB_PATH + ".tmp%d" % os.getpid()
    cmd = ["gcc", "-O2", "-std=c11", "-Wall", "-Wextra", "-fopenmp",
           "-ffp-contract=off", "-fPIC", "-shared", _SRC, "-o", tmp, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB_PATH)
    return LIB_PATH


def build_native(directory: str) -> str:
    """Compile the same source with -O3 -march=native (still no FMA
    contraction, so every result is bit-identical to the portable build) into
    `directory`, for timing the oracle on the host it runs on.  Returns the
    library path."""
    os.makedirs(directory, exist_ok=True)
    path = os.path.join(directory, "libdecode_attn_oracle_native.so")
    cmd = ["gcc", "-O3", "-march=native", "-std=c11", "-Wall", "-Wextra", "-fopenmp",
           "-ffp-contract=off", "-fPIC", "-shared", _SRC, "-o", path, "-lm"]
    subprocess.run(cmd, check=True)
    return path


class using_library:
    """Context manager: oracle calls inside it go to the library at `path`
    (for instance a build_native() build)."""

    def __init__(self, path: str):
        self.path = path
        self.saved = None

    def __enter__(self):
        self.saved = _lib
        _load_path(self.path)
        return self

    def __exit__(self, *exc):
        global _lib
        _lib = self.saved
        return False


class _Append(ctypes.Structure):
    _fields_ = [
        ("batch", ctypes.c_int32),
        ("num_kv_heads", ctypes.c_int32),
        ("head_dim", ctypes.c_int32),
        ("page_size", ctypes.c_int32),
        ("kv_dtype", ctypes.c_int32),
        ("layout", ctypes.c_int32),
        ("max_pages", ctypes.c_int32),
        ("num_pages", ctypes.c_int64),
        ("k_new", ctypes.c_void_p),
        ("v_new", ctypes.c_void_p),
        ("k_pool", ctypes.c_void_p),
        ("v_pool", ctypes.c_void_p),
        ("k_scale", ctypes.c_void_p),
        ("v_scale", ctypes.c_void_p),
        ("block_table", ctypes.c_void_p),
        ("seq_lens", ctypes.c_void_p),
    ]


class _Problem(ctypes.Structure):
    _fields_ = [
        ("batch", ctypes.c_int32),
        ("num_q_heads", ctypes.c_int32),
        ("num_kv_heads", ctypes.c_int32),
        ("head_dim", ctypes.c_int32),
        ("page_size", ctypes.c_int32),
        ("kv_dtype", ctypes.c_int32),
        ("layout", ctypes.c_int32),
        ("max_pages", ctypes.c_int32),
        ("num_pages", ctypes.c_int64),
        ("scale", ctypes.c_double),
        ("q", ctypes.c_void_p),
        ("k_pool", ctypes.c_void_p),
        ("v_pool", ctypes.c_void_p),
        ("k_scale", ctypes.c_void_p),
        ("v_scale", ctypes.c_void_p),
        ("block_table", ctypes.c_void_p),
        ("seq_lens", ctypes.c_void_p),
    ]


_lib = None


def _load():
    global _lib
    if _lib is None:
        # RL_ORACLE_LIB points the tests at a deliberately mutated build of the
        # oracle, to show that the pins catch plausible mistakes.
        path = os.environ.get("RL_ORACLE_LIB") or LIB_PATH
        if path == LIB_PATH and not os.path.exists(LIB_PATH):
            build()
        _load_path(path)
    return _lib


def _load_path(path):
    """Loads the oracle library at `path` as the one later calls use."""
    global _lib
    lib = ctypes.CDLL(path)
    lib.rl_oracle_decode_attn.argtypes = [
        ctypes.POINTER(_Problem), ctypes.c_void_p, ctypes.c_int64,
        ctypes.c_void_p]
    lib.rl_oracle_decode_attn.restype = ctypes.c_int
    lib.rl_oracle_e4m3_to_double.argtypes = [ctypes.c_uint8]
    lib.rl_oracle_e4m3_to_double.restype = ctypes.c_double
    lib.rl_oracle_bf16_to_double.argtypes = [ctypes.c_uint16]
    lib.rl_oracle_bf16_to_double.restype = ctypes.c_double
    lib.rl_oracle_extend_attn.argtypes = [ctypes.POINTER(_Problem), ctypes.c_void_p,
                                          ctypes.c_void_p]
    lib.rl_oracle_extend_attn.restype = ctypes.c_int
    lib.rl_oracle_kv_append.argtypes = [ctypes.POINTER(_Append)]
    lib.rl_oracle_kv_append.restype = ctypes.c_int
    lib.rl_oracle_e4m3_encode.argtypes = [ctypes.c_float]
    lib.rl_oracle_e4m3_encode.restype = ctypes.c_uint8
    lib.rl_oracle_max_threads.argtypes = []
    lib.rl_oracle_max_threads.restype = ctypes.c_int
    _lib = lib
    return _lib


def _layout_code(layout):
    codes = {LAYOUT_HND: LAYOUT_HND, LAYOUT_NHD: LAYOUT_NHD, "hnd": LAYOUT_HND,
             "nhd": LAYOUT_NHD}
    if layout not in codes:
        raise ValueError("unknown pool layout %r" % (layout,))
    return codes[layout]


def _pool_dims(pool, layout):
    """(num_pages, num_kv_heads, page_size, head_dim) of a pool array."""
    if _layout_code(layout) == LAYOUT_NHD:
        P, page, Hkv, D = pool.shape
    else:
        P, Hkv, page, D = pool.shape
    return P, Hkv, page, D


def _c(a, dtype):
    a = np.ascontiguousarray(a)
    if a.dtype != dtype:
        raise TypeError("expected %s, got %s" % (np.dtype(dtype), a.dtype))
    return a


def decode_attention(q_bits, k_pool, v_pool, block_table, seq_lens, *,
                     num_kv_heads, scale, kv_dtype=KV_BF16, k_scale=None,
                     v_scale=None, rows=None, layout=LAYOUT_HND):
    """Attention rows in fp64.

    q_bits      uint16 [B, Hq, D] bf16 bit patterns
    k_pool/v_pool uint16 (bf16 bits) or uint8 (e4m3 codes) [P, Hkv, page, D]
    block_table int32 [B, max_pages];  seq_lens int32 [B]
    rows        None (all (b, h), returns [B, Hq, D]) or int array [n, 2] of
                (b, h) pairs (returns [n, D]).
    """
    lib = _load()
    q_bits = _c(q_bits, np.uint16)
    pool_dtype = np.uint16 if kv_dtype == KV_BF16 else np.uint8
    k_pool = _c(k_pool, pool_dtype)
    v_pool = _c(v_pool, pool_dtype)
    block_table = _c(block_table, np.int32)
    seq_lens = _c(seq_lens, np.int32)
    B, Hq, D = q_bits.shape
    P, Hkv, page, D2 = _pool_dims(k_pool, layout)
    if D2 != D or v_pool.shape != k_pool.shape or Hkv != num_kv_heads:
        raise ValueError("pool shape does not match q / num_kv_heads")
    if block_table.ndim != 2 or block_table.shape[0] != B or seq_lens.shape != (B,):
        raise ValueError("block_table / seq_lens shape")
    if kv_dtype == KV_FP8_E4M3:
        k_scale = _c(k_scale, np.float32)
        v_scale = _c(v_scale, np.float32)
        if k_scale.shape != (P, Hkv) or v_scale.shape != (P, Hkv):
            raise ValueError("scale shape")
    prob = _Problem(
        batch=B, num_q_heads=Hq, num_kv_heads=Hkv, head_dim=D, page_size=page,
        kv_dtype=kv_dtype, layout=_layout_code(layout), max_pages=block_table.shape[1],
        num_pages=P,
        scale=float(scale), q=q_bits.ctypes.data, k_pool=k_pool.ctypes.data,
        v_pool=v_pool.ctypes.data,
        k_scale=k_scale.ctypes.data if kv_dtype == KV_FP8_E4M3 else None,
        v_scale=v_scale.ctypes.data if kv_dtype == KV_FP8_E4M3 else None,
        block_table=block_table.ctypes.data, seq_lens=seq_lens.ctypes.data)
    if rows is None:
        out = np.empty((B, Hq, D), dtype=np.float64)
        rc = lib.rl_oracle_decode_attn(ctypes.byref(prob), None, 0,
                                       out.ctypes.data)
    else:
        rows = _c(np.asarray(rows, dtype=np.int32).reshape(-1, 2), np.int32)
        out = np.empty((rows.shape[0], D), dtype=np.float64)
        rc = lib.rl_oracle_decode_attn(ctypes.byref(prob), rows.ctypes.data,
                                       rows.shape[0], out.ctypes.data)
    if rc != OK:
        raise OracleError("oracle failed with code %d" % rc)
    return out


def extend_attention(q_bits, q_start, k_pool, v_pool, block_table, seq_lens, *,
                     num_kv_heads, scale, kv_dtype=KV_BF16, k_scale=None, v_scale=None,
                     layout=LAYOUT_HND):
    """Causal attention of each sequence's new tokens (q rows q_start[b] ..
    q_start[b+1]-1, the last n_b cached tokens) over its cache.  q_bits uint16
    [T, Hq, D]; returns fp64 [T, Hq, D]."""
    lib = _load()
    q_bits = _c(q_bits, np.uint16)
    q_start = _c(q_start, np.int32)
    pool_dtype = np.uint16 if kv_dtype == KV_BF16 else np.uint8
    k_pool = _c(k_pool, pool_dtype)
    v_pool = _c(v_pool, pool_dtype)
    block_table = _c(block_table, np.int32)
    seq_lens = _c(seq_lens, np.int32)
    T, Hq, D = q_bits.shape
    B = seq_lens.shape[0]
    P, Hkv, page, _ = _pool_dims(k_pool, layout)
    if q_start.shape != (B + 1,) or q_start[-1] != T:
        raise ValueError("q_start must have batch+1 entries ending at T")
    if kv_dtype == KV_FP8_E4M3:
        k_scale = _c(k_scale, np.float32)
        v_scale = _c(v_scale, np.float32)
    prob = _Problem(
        batch=B, num_q_heads=Hq, num_kv_heads=Hkv, head_dim=D, page_size=page,
        kv_dtype=kv_dtype, layout=_layout_code(layout), max_pages=block_table.shape[1],
        num_pages=P,
        scale=float(scale), q=q_bits.ctypes.data, k_pool=k_pool.ctypes.data,
        v_pool=v_pool.ctypes.data,
        k_scale=k_scale.ctypes.data if kv_dtype == KV_FP8_E4M3 else None,
        v_scale=v_scale.ctypes.data if kv_dtype == KV_FP8_E4M3 else None,
        block_table=block_table.ctypes.data, seq_lens=seq_lens.ctypes.data)
    out = np.empty((T, Hq, D), dtype=np.float64)
    rc = lib.rl_oracle_extend_attn(ctypes.byref(prob), q_start.ctypes.data, out.ctypes.data)
    if rc != OK:
        raise OracleError("oracle extend failed with code %d" % rc)
    return out


def kv_append(k_new_bits, v_new_bits, k_pool, v_pool, block_table, seq_lens, *,
              kv_dtype=KV_BF16, k_scale=None, v_scale=None, layout=LAYOUT_HND):
    """Appends one token per (sequence, kv head); returns updated copies of
    (k_pool, v_pool, k_scale, v_scale).  k_new/v_new: uint16 bf16 bits
    [B, Hkv, D]; pools as in decode_attention; seq_lens = lengths before the
    append."""
    lib = _load()
    k_new_bits = _c(k_new_bits, np.uint16)
    v_new_bits = _c(v_new_bits, np.uint16)
    pool_dtype = np.uint16 if kv_dtype == KV_BF16 else np.uint8
    k_pool = _c(k_pool, pool_dtype).copy()
    v_pool = _c(v_pool, pool_dtype).copy()
    block_table = _c(block_table, np.int32)
    seq_lens = _c(seq_lens, np.int32)
    B, Hkv, D = k_new_bits.shape
    P, Hkv2, page, D2 = _pool_dims(k_pool, layout)
    if (Hkv2, D2) != (Hkv, D) or v_new_bits.shape != k_new_bits.shape:
        raise ValueError("shape mismatch")
    if kv_dtype == KV_FP8_E4M3:
        k_scale = _c(k_scale, np.float32).copy()
        v_scale = _c(v_scale, np.float32).copy()
    prob = _Append(
        batch=B, num_kv_heads=Hkv, head_dim=D, page_size=page, kv_dtype=kv_dtype,
        layout=_layout_code(layout), max_pages=block_table.shape[1], num_pages=P, k_new=k_new_bits.ctypes.data,
        v_new=v_new_bits.ctypes.data, k_pool=k_pool.ctypes.data, v_pool=v_pool.ctypes.data,
        k_scale=k_scale.ctypes.data if kv_dtype == KV_FP8_E4M3 else None,
        v_scale=v_scale.ctypes.data if kv_dtype == KV_FP8_E4M3 else None,
        block_table=block_table.ctypes.data, seq_lens=seq_lens.ctypes.data)
    rc = lib.rl_oracle_kv_append(ctypes.byref(prob))
    if rc != OK:
        raise OracleError("oracle append failed with code %d" % rc)
    return k_pool, v_pool, k_scale, v_scale


def e4m3_encode(x: float) -> int:
    return _load().rl_oracle_e4m3_encode(float(x))


def e4m3_to_double(code: int) -> float:
    return _load().rl_oracle_e4m3_to_double(int(code))


def bf16_to_double(bits: int) -> float:
    return _load().rl_oracle_bf16_to_double(int(bits))


def max_threads() -> int:
    return _load().rl_oracle_max_threads()


def set_threads(n: int) -> None:
    """Threads for later oracle calls (OpenMP)."""
    lib = _load()
    lib.rl_oracle_set_threads.argtypes = [ctypes.c_int]
    lib.rl_oracle_set_threads.restype = None
    lib.rl_oracle_set_threads(int(n))
