"""ctypes binding of the C interface declared in include/rl_decode_attn.h.

Argument marshalling only: every step of the attention runs in the HIP
library.  Functions keep the C names.  Pointer arguments accept either an
integer device address or a torch tensor (its data_ptr is passed); `stream`
accepts an integer hipStream_t, a torch.cuda.Stream or None (null stream).
The library is loaded on first use and a missing build is an error.
"""
from __future__ import annotations

import ctypes
import os

from . import build as _build

RL_DA_OK = 0
RL_DA_ERR_INVALID_ARG = 1
RL_DA_ERR_UNSUPPORTED = 2
RL_DA_ERR_OUT_OF_MEMORY = 3
RL_DA_ERR_HIP = 4
RL_DA_ERR_SCRATCH_TOO_SMALL = 5
RL_DA_NOALLOC_SCRATCH_BYTES = 64 << 20

RL_DA_KV_BF16 = 0
RL_DA_KV_FP8_E4M3 = 1
KV_DTYPES = {"bf16": RL_DA_KV_BF16, "fp8_e4m3": RL_DA_KV_FP8_E4M3}

RL_DA_LAYOUT_HND = 0
RL_DA_LAYOUT_NHD = 1
RL_DA_LAYOUT_HND_KV = 2
LAYOUTS = {"hnd": RL_DA_LAYOUT_HND, "nhd": RL_DA_LAYOUT_NHD, "hnd_kv": RL_DA_LAYOUT_HND_KV}

RL_DA_CHECKED = 0x1
RL_DA_SCORES_ON_VALU = 0x2
RL_DA_PER_HEAD_UNITS = 0x4
RL_DA_PV_ON_VALU = 0x8

RL_DA_DEVERR_PAGE_OUT_OF_RANGE = 0x1
RL_DA_DEVERR_LENGTH_TOO_LONG = 0x2

# Every function the header declares, in declaration order.
EXPORTED = [
    "rl_decode_attn_create",
    "rl_decode_attn_run",
    "rl_decode_attn_destroy",
    "rl_da_status_string",
    "rl_decode_attn_workspace_size",
    "rl_decode_attn_check_error",
    "rl_decode_attn_split_info",
    "rl_decode_attn_unit_heads",
    "rl_extend_attn",
    "rl_kv_append",
    "rl_decode_attn_set_timing_events",
    "rl_ws_plan",
    "rl_ws_create",
    "rl_ws_num_chunks",
    "rl_ws_chunk_bytes",
    "rl_ws_pack",
    "rl_ws_unpack",
    "rl_ws_destroy",
    "rl_decode_attn_run_noalloc",
]


class rl_da_config(ctypes.Structure):
    _fields_ = [
        ("num_q_heads", ctypes.c_int32),
        ("num_kv_heads", ctypes.c_int32),
        ("head_dim", ctypes.c_int32),
        ("page_size", ctypes.c_int32),
        ("max_batch", ctypes.c_int32),
        ("max_pages_per_seq", ctypes.c_int32),
        ("kv_dtype", ctypes.c_int32),
        ("layout", ctypes.c_int32),
        ("split_tokens", ctypes.c_int32),
        ("flags", ctypes.c_uint32),
    ]


class rl_ws_tensor(ctypes.Structure):
    _fields_ = [("ptr", ctypes.c_void_p), ("nbytes", ctypes.c_uint64)]


class rl_ws_piece(ctypes.Structure):
    _fields_ = [
        ("tensor", ctypes.c_int32),
        ("chunk", ctypes.c_int32),
        ("tensor_offset", ctypes.c_uint64),
        ("buffer_offset", ctypes.c_uint64),
        ("nbytes", ctypes.c_uint64),
    ]


class RLDecodeAttnError(RuntimeError):
    def __init__(self, status: int, what: str):
        super().__init__("%s failed: %s (status %d)" % (what, _status_text(status), status))
        self.status = status


_lib = None


def library_path() -> str:
    return _build.LIB_PATH


def load_library():
    """Loads the built library; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    path = _build.LIB_PATH
    if not os.path.exists(path):
        raise RuntimeError(
            "HIP library %s is not built; run __graft_entry__.build()" % path)
    # torch carries its own HIP runtime under the same soname
    # (libamdhip64.so.7).  Loading torch first makes the library bind to that
    # one copy, so device pointers, streams and events are shared; loading it
    # first would pull a second runtime into the process.
    import torch  # noqa: F401
    lib = ctypes.CDLL(path)
    vp, i32, i64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
    lib.rl_decode_attn_create.argtypes = [ctypes.POINTER(rl_da_config), ctypes.POINTER(vp)]
    lib.rl_decode_attn_create.restype = ctypes.c_int
    lib.rl_decode_attn_run.argtypes = [vp, vp, vp, vp, vp, vp, i64, vp, i32, vp, i32,
                                       ctypes.c_float, vp, vp]
    lib.rl_decode_attn_run.restype = ctypes.c_int
    lib.rl_decode_attn_run_noalloc.argtypes = [ctypes.POINTER(rl_da_config), vp, vp, vp, vp,
                                               vp, i64, vp, i32, vp, i32, ctypes.c_float, vp,
                                               vp]
    lib.rl_decode_attn_run_noalloc.restype = ctypes.c_int
    lib.rl_decode_attn_destroy.argtypes = [vp]
    lib.rl_decode_attn_destroy.restype = ctypes.c_int
    lib.rl_da_status_string.argtypes = [ctypes.c_int]
    lib.rl_da_status_string.restype = ctypes.c_char_p
    lib.rl_decode_attn_workspace_size.argtypes = [ctypes.POINTER(rl_da_config),
                                                  ctypes.POINTER(ctypes.c_size_t)]
    lib.rl_decode_attn_workspace_size.restype = ctypes.c_int
    lib.rl_decode_attn_check_error.argtypes = [vp, ctypes.POINTER(i32)]
    lib.rl_decode_attn_check_error.restype = ctypes.c_int
    lib.rl_decode_attn_split_info.argtypes = [vp, i32, ctypes.POINTER(i32), ctypes.POINTER(i32)]
    lib.rl_decode_attn_split_info.restype = ctypes.c_int
    lib.rl_decode_attn_unit_heads.argtypes = [vp, ctypes.POINTER(i32)]
    lib.rl_decode_attn_unit_heads.restype = ctypes.c_int
    lib.rl_extend_attn.argtypes = [vp, vp, i32, vp, vp, vp, vp, i64, vp, i32, vp, i32, i32, i32,
                                   i32, i32, i32, i32, ctypes.c_float, vp, vp]
    lib.rl_extend_attn.restype = ctypes.c_int
    lib.rl_kv_append.argtypes = [vp, vp, vp, vp, vp, vp, i64, vp, i32, vp, i32, i32, i32, i32,
                                 i32, i32, vp, vp]
    lib.rl_kv_append.restype = ctypes.c_int
    lib.rl_decode_attn_set_timing_events.argtypes = [vp, vp, vp]
    lib.rl_decode_attn_set_timing_events.restype = ctypes.c_int
    u64 = ctypes.c_uint64
    lib.rl_ws_plan.argtypes = [ctypes.POINTER(u64), i32, u64, u64, ctypes.POINTER(rl_ws_piece),
                               i64, ctypes.POINTER(i64), ctypes.POINTER(i32)]
    lib.rl_ws_plan.restype = ctypes.c_int
    lib.rl_ws_create.argtypes = [ctypes.POINTER(rl_ws_tensor), i32, vp, u64, u64,
                                 ctypes.POINTER(vp)]
    lib.rl_ws_create.restype = ctypes.c_int
    lib.rl_ws_num_chunks.argtypes = [vp, ctypes.POINTER(i32)]
    lib.rl_ws_num_chunks.restype = ctypes.c_int
    lib.rl_ws_chunk_bytes.argtypes = [vp, i32, ctypes.POINTER(u64)]
    lib.rl_ws_chunk_bytes.restype = ctypes.c_int
    lib.rl_ws_pack.argtypes = [vp, i32, vp]
    lib.rl_ws_pack.restype = ctypes.c_int
    lib.rl_ws_unpack.argtypes = [vp, i32, vp]
    lib.rl_ws_unpack.restype = ctypes.c_int
    lib.rl_ws_destroy.argtypes = [vp]
    lib.rl_ws_destroy.restype = ctypes.c_int
    _lib = lib
    return lib


def _status_text(status: int) -> str:
    try:
        return load_library().rl_da_status_string(status).decode()
    except Exception:
        return "status %d" % status


def _ptr(x):
    if x is None:
        return None
    if isinstance(x, int):
        return x
    return x.data_ptr()


def _stream(s):
    if s is None:
        return None
    if isinstance(s, int):
        return s
    return s.cuda_stream


def _pool_shape(layout, num_pages, num_kv_heads, page_size, head_dim):
    if layout == "nhd":
        return (num_pages, page_size, num_kv_heads, head_dim)
    return (num_pages, num_kv_heads, page_size, head_dim)


def _check_tensor(name, t, *, dtype=None, shape=None, ndim=None, device=None,
                  contiguous=True):
    """Raises ValueError unless t is a (contiguous) torch tensor of the given
    dtype, shape (None entries match anything) and device."""
    # called on every entry point's every tensor: the common case (exact
    # dtype, exact shape) takes the cheap comparisons first
    if not hasattr(t, "data_ptr") or not hasattr(t, "is_contiguous"):
        raise ValueError("%s must be a torch tensor" % name)
    if dtype is not None and t.dtype != dtype and (not isinstance(dtype, tuple)
                                                   or t.dtype not in dtype):
        raise ValueError("%s has dtype %s, expected %s" % (name, t.dtype, dtype))
    if contiguous and not t.is_contiguous():
        raise ValueError("%s must be contiguous" % name)
    if ndim is not None and t.dim() != ndim:
        raise ValueError("%s must have %d dimensions, has shape %s" % (name, ndim, tuple(t.shape)))
    if shape is not None:
        ts = tuple(t.shape)
        if ts != tuple(shape) and (len(ts) != len(shape) or any(
                w is not None and d != w for d, w in zip(ts, shape))):
            raise ValueError("%s has shape %s, expected %s"
                             % (name, ts, tuple("*" if w is None else w for w in shape)))
    if device is not None and t.device != device:
        raise ValueError("%s is on %s, expected %s" % (name, t.device, device))


def _check_pools(k_pool, v_pool, k_scale, v_scale, *, kv_dtype, layout, num_kv_heads,
                 head_dim, page_size, device):
    """The pools' dtype (bf16 or uint8 e4m3 codes), layout shape and device;
    fp32 [num_pages, num_kv_heads] scales exactly for e4m3.  Returns num_pages."""
    import torch
    elt = torch.bfloat16 if kv_dtype == RL_DA_KV_BF16 else torch.uint8
    paired = layout == RL_DA_LAYOUT_HND_KV
    _check_tensor("k_pool", k_pool, dtype=elt, ndim=4, device=device, contiguous=not paired)
    P = int(k_pool.shape[0])
    want = _pool_shape("nhd" if layout == RL_DA_LAYOUT_NHD else "hnd", P, num_kv_heads,
                       page_size, head_dim)
    _check_tensor("k_pool", k_pool, shape=want, contiguous=not paired)
    _check_tensor("v_pool", v_pool, dtype=elt, shape=want, device=device,
                  contiguous=not paired)
    if paired:
        # views of one [P, Hkv, 2, page, D] allocation: key slab, then value slab
        slab = page_size * head_dim
        strides = (num_kv_heads * 2 * slab, 2 * slab, head_dim, 1)
        if tuple(k_pool.stride()) != strides or tuple(v_pool.stride()) != strides:
            raise ValueError("hnd_kv pools must be the [:, :, 0] and [:, :, 1] views of one "
                             "contiguous [P, Hkv, 2, page, D] tensor")
        if v_pool.data_ptr() != k_pool.data_ptr() + slab * k_pool.element_size():
            raise ValueError("hnd_kv: v_pool must start one slab after k_pool")
    if kv_dtype == RL_DA_KV_BF16:
        if k_scale is not None or v_scale is not None:
            raise ValueError("bf16 pools take no k_scale / v_scale")
    else:
        _check_tensor("k_scale", k_scale, dtype=torch.float32, shape=(P, num_kv_heads),
                      device=device)
        _check_tensor("v_scale", v_scale, dtype=torch.float32, shape=(P, num_kv_heads),
                      device=device)
    return P


def _check_table(block_table, seq_lens, batch, device):
    import torch
    _check_tensor("block_table", block_table, dtype=torch.int32, ndim=2, device=device)
    if int(block_table.shape[0]) != batch:
        raise ValueError("block_table has %d rows for a batch of %d"
                         % (block_table.shape[0], batch))
    _check_tensor("seq_lens", seq_lens, dtype=torch.int32, shape=(batch,), device=device)


def make_config(num_q_heads, num_kv_heads, max_batch, max_pages_per_seq, *,
                head_dim=128, page_size=16, kv_dtype=RL_DA_KV_BF16,
                layout=RL_DA_LAYOUT_HND, split_tokens=0, flags=0) -> rl_da_config:
    return rl_da_config(num_q_heads=num_q_heads, num_kv_heads=num_kv_heads,
                        head_dim=head_dim, page_size=page_size, max_batch=max_batch,
                        max_pages_per_seq=max_pages_per_seq, kv_dtype=kv_dtype,
                        layout=layout, split_tokens=split_tokens, flags=flags)


# ------------------------------------------------- C functions, same names ---

def rl_da_status_string(status: int) -> str:
    return load_library().rl_da_status_string(int(status)).decode()


def rl_decode_attn_create(cfg: rl_da_config):
    """Returns (status, handle); handle is None unless status is RL_DA_OK."""
    h = ctypes.c_void_p()
    rc = load_library().rl_decode_attn_create(ctypes.byref(cfg), ctypes.byref(h))
    return rc, (h.value if rc == RL_DA_OK else None)


def rl_decode_attn_run(h, q, k_pool, v_pool, k_scale, v_scale, num_pages, block_table,
                       max_pages, seq_lens, batch, scale, out, stream=None) -> int:
    return load_library().rl_decode_attn_run(
        h, _ptr(q), _ptr(k_pool), _ptr(v_pool), _ptr(k_scale), _ptr(v_scale),
        int(num_pages), _ptr(block_table), int(max_pages), _ptr(seq_lens), int(batch),
        float(scale), _ptr(out), _stream(stream))


def rl_decode_attn_run_noalloc(cfg, q, k_pool, v_pool, k_scale, v_scale, num_pages,
                               block_table, max_pages, seq_lens, batch, scale, out,
                               stream=None) -> int:
    return load_library().rl_decode_attn_run_noalloc(
        ctypes.byref(cfg), _ptr(q), _ptr(k_pool), _ptr(v_pool), _ptr(k_scale), _ptr(v_scale),
        int(num_pages), _ptr(block_table), int(max_pages), _ptr(seq_lens), int(batch),
        float(scale), _ptr(out), _stream(stream))


def rl_decode_attn_destroy(h) -> int:
    return load_library().rl_decode_attn_destroy(h)


def rl_decode_attn_workspace_size(cfg: rl_da_config):
    n = ctypes.c_size_t()
    rc = load_library().rl_decode_attn_workspace_size(ctypes.byref(cfg), ctypes.byref(n))
    return rc, n.value


def rl_decode_attn_check_error(h):
    v = ctypes.c_int32()
    rc = load_library().rl_decode_attn_check_error(h, ctypes.byref(v))
    return rc, v.value


def rl_decode_attn_split_info(h, max_pages):
    st, ns = ctypes.c_int32(), ctypes.c_int32()
    rc = load_library().rl_decode_attn_split_info(h, int(max_pages), ctypes.byref(st),
                                                  ctypes.byref(ns))
    return rc, st.value, ns.value


def rl_decode_attn_unit_heads(h):
    v = ctypes.c_int32()
    rc = load_library().rl_decode_attn_unit_heads(h, ctypes.byref(v))
    return rc, v.value


def rl_extend_attn(q, q_start, max_q_per_seq, k_pool, v_pool, k_scale, v_scale, num_pages,
                   block_table, max_pages, seq_lens, batch, num_q_heads, num_kv_heads,
                   head_dim=128, page_size=16, kv_dtype=RL_DA_KV_BF16, layout=RL_DA_LAYOUT_HND,
                   scale=1.0, out=None, stream=None) -> int:
    return load_library().rl_extend_attn(
        _ptr(q), _ptr(q_start), int(max_q_per_seq), _ptr(k_pool), _ptr(v_pool), _ptr(k_scale),
        _ptr(v_scale), int(num_pages), _ptr(block_table), int(max_pages), _ptr(seq_lens),
        int(batch), int(num_q_heads), int(num_kv_heads), int(head_dim), int(page_size),
        int(kv_dtype), int(layout), float(scale), _ptr(out), _stream(stream))


def extend_attention(p, q, q_start, max_q_per_seq, out, stream=None):
    """Extend attention of new tokens q [T, Hq, D] (rows q_start[b]..) over
    problem p's cache (p.seq_lens include the new tokens); raises on error."""
    import torch
    dt = RL_DA_KV_BF16 if p.kv_dtype == "bf16" else RL_DA_KV_FP8_E4M3
    dev = p.k_pool.device
    _check_tensor("q", q, dtype=torch.bfloat16, shape=(None, p.num_q_heads, p.head_dim),
                  device=dev)
    _check_tensor("out", out, dtype=torch.bfloat16, shape=tuple(q.shape), device=dev)
    _check_tensor("q_start", q_start, dtype=torch.int32, shape=(p.batch + 1,), device=dev)
    _check_pools(p.k_pool, p.v_pool, p.k_scale, p.v_scale, kv_dtype=dt,
                 layout=LAYOUTS[p.layout], num_kv_heads=p.num_kv_heads, head_dim=p.head_dim,
                 page_size=p.page_size, device=dev)
    _check_table(p.block_table, p.seq_lens, p.batch, dev)
    rc = rl_extend_attn(q, q_start, max_q_per_seq, p.k_pool, p.v_pool, p.k_scale, p.v_scale,
                        p.num_pages, p.block_table, p.max_pages, p.seq_lens, p.batch,
                        p.num_q_heads, p.num_kv_heads, p.head_dim, p.page_size, dt,
                        LAYOUTS[p.layout], p.scale, out, stream)
    if rc != RL_DA_OK:
        raise RLDecodeAttnError(rc, "rl_extend_attn")


def rl_kv_append(k_new, v_new, k_pool, v_pool, k_scale, v_scale, num_pages, block_table,
                 max_pages, seq_lens, batch, num_kv_heads, head_dim=128, page_size=16,
                 kv_dtype=RL_DA_KV_BF16, layout=RL_DA_LAYOUT_HND, device_error=None,
                 stream=None) -> int:
    return load_library().rl_kv_append(
        _ptr(k_new), _ptr(v_new), _ptr(k_pool), _ptr(v_pool), _ptr(k_scale), _ptr(v_scale),
        int(num_pages), _ptr(block_table), int(max_pages), _ptr(seq_lens), int(batch),
        int(num_kv_heads), int(head_dim), int(page_size), int(kv_dtype), int(layout),
        _ptr(device_error), _stream(stream))


class KvAppender:
    """rl_kv_append for a loop that appends to one cache step after step:
    checks problem p's pools, scales, block table and lengths once, here, and
    only the new tokens on each call.  Those cache tensors must keep their
    storage, dtype and shape while the appender is used (their contents may
    change: the table and lengths are read by the kernel on every call)."""

    def __init__(self, p, device_error=None):
        import torch
        self.kv_dtype = RL_DA_KV_BF16 if p.kv_dtype == "bf16" else RL_DA_KV_FP8_E4M3
        self.device = p.k_pool.device
        self.want = (p.batch, p.num_kv_heads, p.head_dim)
        _check_pools(p.k_pool, p.v_pool, p.k_scale, p.v_scale, kv_dtype=self.kv_dtype,
                     layout=LAYOUTS[p.layout], num_kv_heads=p.num_kv_heads,
                     head_dim=p.head_dim, page_size=p.page_size, device=self.device)
        _check_table(p.block_table, p.seq_lens, p.batch, self.device)
        if device_error is not None:
            _check_tensor("device_error", device_error, dtype=torch.int32, device=self.device)
        self._fn = load_library().rl_kv_append
        self._cache_args = (
            _ptr(p.k_pool), _ptr(p.v_pool), _ptr(p.k_scale), _ptr(p.v_scale),
            int(p.num_pages), _ptr(p.block_table), int(p.max_pages), _ptr(p.seq_lens),
            int(p.batch), int(p.num_kv_heads), int(p.head_dim), int(p.page_size),
            int(self.kv_dtype), int(LAYOUTS[p.layout]), _ptr(device_error))

    def __call__(self, k_new, v_new, stream=None):
        """Appends k_new/v_new [B, Hkv, D] (bf16) at positions seq_lens;
        raises on a bad status."""
        import torch
        _check_tensor("k_new", k_new, dtype=torch.bfloat16, shape=self.want, device=self.device)
        _check_tensor("v_new", v_new, dtype=torch.bfloat16, shape=self.want, device=self.device)
        rc = self._fn(k_new.data_ptr(), v_new.data_ptr(), *self._cache_args, _stream(stream))
        if rc != RL_DA_OK:
            raise RLDecodeAttnError(rc, "rl_kv_append")


def kv_append(p, k_new, v_new, device_error=None, stream=None):
    """Appends k_new/v_new [B, Hkv, D] (bf16 tensors) to problem p's pools at
    positions p.seq_lens; raises on a bad status."""
    KvAppender(p, device_error)(k_new, v_new, stream)


def rl_decode_attn_set_timing_events(h, split_begin, split_end) -> int:
    return load_library().rl_decode_attn_set_timing_events(h, split_begin, split_end)


def rl_ws_plan(tensor_bytes, capacity, align):
    """Returns (status, pieces as (tensor, chunk, tensor_offset, buffer_offset,
    nbytes) tuples, num_chunks)."""
    lib = load_library()
    n = len(tensor_bytes)
    sizes = (ctypes.c_uint64 * max(1, n))(*[int(x) for x in tensor_bytes])
    np_, nc = ctypes.c_int64(), ctypes.c_int32()
    rc = lib.rl_ws_plan(sizes, n, int(capacity), int(align), None, 0, ctypes.byref(np_),
                        ctypes.byref(nc))
    if rc != RL_DA_OK:
        return rc, None, None
    buf = (rl_ws_piece * max(1, np_.value))()
    rc = lib.rl_ws_plan(sizes, n, int(capacity), int(align), buf, np_.value,
                        ctypes.byref(np_), ctypes.byref(nc))
    pieces = [(p.tensor, p.chunk, p.tensor_offset, p.buffer_offset, p.nbytes)
              for p in buf[:np_.value]]
    return rc, pieces, nc.value


def rl_ws_create(tensors, buffer, capacity, align):
    """tensors: sequence of (device address, nbytes).  Returns (status, handle)."""
    arr = (rl_ws_tensor * max(1, len(tensors)))(
        *[rl_ws_tensor(_ptr(p) if not isinstance(p, int) else p, int(n)) for p, n in tensors])
    h = ctypes.c_void_p()
    rc = load_library().rl_ws_create(arr, len(tensors), _ptr(buffer), int(capacity), int(align),
                                     ctypes.byref(h))
    return rc, (h.value if rc == RL_DA_OK else None)


def rl_ws_num_chunks(h):
    n = ctypes.c_int32()
    rc = load_library().rl_ws_num_chunks(h, ctypes.byref(n))
    return rc, n.value


def rl_ws_chunk_bytes(h, chunk):
    n = ctypes.c_uint64()
    rc = load_library().rl_ws_chunk_bytes(h, int(chunk), ctypes.byref(n))
    return rc, n.value


def rl_ws_pack(h, chunk, stream=None) -> int:
    return load_library().rl_ws_pack(h, int(chunk), _stream(stream))


def rl_ws_unpack(h, chunk, stream=None) -> int:
    return load_library().rl_ws_unpack(h, int(chunk), _stream(stream))


def rl_ws_destroy(h) -> int:
    return load_library().rl_ws_destroy(h)


class WeightSync:
    """Owns one packing plan: tensors (torch tensors on the GPU, packed as raw
    bytes in list order) and a transfer buffer (a uint8 tensor on the GPU or in
    pinned host memory)."""

    def __init__(self, tensors, buffer, align=256):
        for t in tensors:
            if not t.is_contiguous():
                raise ValueError("tensors must be contiguous")
        self.tensors = list(tensors)
        self.buffer = buffer
        spec = [(t.data_ptr(), t.numel() * t.element_size()) for t in self.tensors]
        rc, h = rl_ws_create(spec, buffer, buffer.numel() * buffer.element_size(), align)
        if rc != RL_DA_OK:
            raise RLDecodeAttnError(rc, "rl_ws_create")
        self.handle = h
        rc, self.num_chunks = rl_ws_num_chunks(h)
        if rc != RL_DA_OK:
            raise RLDecodeAttnError(rc, "rl_ws_num_chunks")

    def chunk_bytes(self, chunk):
        rc, n = rl_ws_chunk_bytes(self.handle, chunk)
        if rc != RL_DA_OK:
            raise RLDecodeAttnError(rc, "rl_ws_chunk_bytes")
        return n

    def pack(self, chunk, stream=None):
        rc = rl_ws_pack(self.handle, chunk, stream)
        if rc != RL_DA_OK:
            raise RLDecodeAttnError(rc, "rl_ws_pack")

    def unpack(self, chunk, stream=None):
        rc = rl_ws_unpack(self.handle, chunk, stream)
        if rc != RL_DA_OK:
            raise RLDecodeAttnError(rc, "rl_ws_unpack")

    def close(self):
        if self.handle is not None:
            rl_ws_destroy(self.handle)
            self.handle = None

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


# --------------------------------------------------------- handle wrapper ---

class DecodeAttention:
    """Owns one library handle; run() enqueues one decode step."""

    def __init__(self, num_q_heads, num_kv_heads, max_batch, max_pages_per_seq, *,
                 kv_dtype="bf16", layout="hnd", split_tokens=0, flags=0, head_dim=128,
                 page_size=16):
        dt = KV_DTYPES[kv_dtype]
        self.kv_dtype = kv_dtype
        self.layout = layout
        self.cfg = make_config(num_q_heads, num_kv_heads, max_batch, max_pages_per_seq,
                               head_dim=head_dim, page_size=page_size, kv_dtype=dt,
                               layout=LAYOUTS[layout], split_tokens=split_tokens, flags=flags)
        rc, h = rl_decode_attn_create(self.cfg)
        if rc != RL_DA_OK:
            raise RLDecodeAttnError(rc, "rl_decode_attn_create")
        self.handle = h
        import torch
        # the library creates the handle on the current device
        self.device = torch.device("cuda", torch.cuda.current_device())

    @classmethod
    def for_problem(cls, p, **kw):
        return cls(p.num_q_heads, p.num_kv_heads, p.batch, p.max_pages,
                   kv_dtype=p.kv_dtype, layout=p.layout, **kw)

    def run(self, q, k_pool, v_pool, k_scale, v_scale, block_table, seq_lens, scale, out,
            stream=None):
        """Checks every tensor (dtype, contiguity, device, shapes that agree
        with the handle) before the C call; raises ValueError otherwise."""
        import torch
        c = self.cfg
        dev = self.device
        _check_tensor("q", q, dtype=torch.bfloat16, shape=(None, c.num_q_heads, c.head_dim),
                      device=dev)
        _check_tensor("out", out, dtype=torch.bfloat16, shape=tuple(q.shape), device=dev)
        _check_pools(k_pool, v_pool, k_scale, v_scale, kv_dtype=c.kv_dtype, layout=c.layout,
                     num_kv_heads=c.num_kv_heads, head_dim=c.head_dim,
                     page_size=c.page_size, device=dev)
        _check_table(block_table, seq_lens, int(q.shape[0]), dev)
        rc = rl_decode_attn_run(self.handle, q, k_pool, v_pool, k_scale, v_scale,
                                k_pool.shape[0], block_table, block_table.shape[1],
                                seq_lens, q.shape[0], scale, out, stream)
        if rc != RL_DA_OK:
            raise RLDecodeAttnError(rc, "rl_decode_attn_run")

    def run_problem(self, p, out, stream=None):
        if p.layout != self.layout:
            raise ValueError("problem layout %r, handle layout %r" % (p.layout, self.layout))
        self.run(p.q, p.k_pool, p.v_pool, p.k_scale, p.v_scale, p.block_table, p.seq_lens,
                 p.scale, out, stream)

    def split_info(self, max_pages):
        rc, st, ns = rl_decode_attn_split_info(self.handle, max_pages)
        if rc != RL_DA_OK:
            raise RLDecodeAttnError(rc, "rl_decode_attn_split_info")
        return st, ns

    def unit_heads(self):
        """kv heads per work unit: 1 (four-wavefront units) or a head group."""
        rc, v = rl_decode_attn_unit_heads(self.handle)
        if rc != RL_DA_OK:
            raise RLDecodeAttnError(rc, "rl_decode_attn_unit_heads")
        return v

    def check_error(self):
        rc, v = rl_decode_attn_check_error(self.handle)
        if rc != RL_DA_OK:
            raise RLDecodeAttnError(rc, "rl_decode_attn_check_error")
        return v

    def close(self):
        if self.handle is not None:
            rl_decode_attn_destroy(self.handle)
            self.handle = None

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
