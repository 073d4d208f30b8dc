"""ctypes binding of libmilo.so (C ABI: include/milo.h).

Argument marshalling only: every step of the computation runs in the library's
HIP kernels.  Device buffers are torch tensors (or raw device addresses as int);
the library is required - there is no fallback, and a missing library raises.
"""
from __future__ import annotations

import ctypes
import os
from typing import Sequence

import numpy as np

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libmilo.so")

MILO_OK = 0
MILO_ERR_INVALID_ARG = -1
MILO_ERR_OUT_OF_MEMORY = -2
MILO_ERR_HIP = -3
MILO_ERR_UNSUPPORTED = -4

_c_i32p = ctypes.POINTER(ctypes.c_int32)
_c_u16p = ctypes.POINTER(ctypes.c_uint16)


class milo_cache_desc(ctypes.Structure):
    _fields_ = [("n_blocks", ctypes.c_int32), ("n_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("block_tokens", _c_i32p),
                ("rank_k", _c_i32p), ("rank_v", _c_i32p)]


class MiloError(RuntimeError):
    def __init__(self, code: int, message: str):
        super().__init__(f"milo error {code}: {message}")
        self.code = code


_lib = None


def lib() -> ctypes.CDLL:
    """Load libmilo.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built: run __graft_entry__.build()")
        # PyTorch ships its own HIP runtime; loading it first makes the library
        # bind to that same runtime (one runtime per process), so torch tensors
        # and streams can be passed across the boundary
        import torch  # noqa: F401
        L = ctypes.CDLL(LIB_PATH)
        vp = ctypes.c_void_p
        L.milo_cache_create.argtypes = [ctypes.POINTER(milo_cache_desc), ctypes.POINTER(vp),
                                        ctypes.POINTER(vp), ctypes.POINTER(vp), ctypes.POINTER(vp),
                                        ctypes.c_int, vp, ctypes.POINTER(vp)]
        L.milo_cache_create.restype = ctypes.c_int
        L.milo_attend_decode.argtypes = [vp, _c_i32p, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                                         vp, vp, vp, _c_i32p, ctypes.c_int32, ctypes.c_float, vp, vp]
        L.milo_attend_decode.restype = ctypes.c_int
        L.milo_attend_prefill.argtypes = [vp, _c_i32p, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                                          vp, vp, vp, ctypes.c_int32, ctypes.c_int32, ctypes.c_float, vp, vp]
        L.milo_attend_prefill.restype = ctypes.c_int
        L.milo_allocate_ranks.argtypes = [vp, ctypes.c_int64, ctypes.c_int32, _c_i32p, ctypes.c_int64,
                                          ctypes.c_int32, ctypes.c_int32, _c_i32p, vp]
        L.milo_allocate_ranks.restype = ctypes.c_int
        L.milo_timing_read_alloc.argtypes = [ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_double),
                                             ctypes.POINTER(ctypes.c_int64)]
        L.milo_timing_read_alloc.restype = ctypes.c_int
        L.milo_cache_free.argtypes = [vp]
        L.milo_cache_free.restype = None
        L.milo_last_error.argtypes = []
        L.milo_last_error.restype = ctypes.c_char_p
        L.milo_cache_device_bytes.argtypes = [vp, ctypes.POINTER(ctypes.c_int64)]
        L.milo_cache_device_bytes.restype = ctypes.c_int
        L.milo_cache_read_factor.argtypes = [vp, ctypes.c_int32, ctypes.c_int32, vp]
        L.milo_cache_read_factor.restype = ctypes.c_int
        L.milo_timing_enable.argtypes = [ctypes.c_int]
        L.milo_timing_enable.restype = ctypes.c_int
        L.milo_timing_read.argtypes = [ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_double),
                                       ctypes.POINTER(ctypes.c_int64)]
        L.milo_timing_read.restype = ctypes.c_int
        _lib = L
    return _lib


def milo_last_error() -> str:
    return lib().milo_last_error().decode()


def _check(code: int) -> None:
    if code != MILO_OK:
        raise MiloError(code, milo_last_error())


def _addr(x) -> int:
    """Address of a torch tensor, numpy array or raw int (None -> 0)."""
    if x is None:
        return 0
    if isinstance(x, int):
        return x
    if isinstance(x, np.ndarray):
        return x.ctypes.data
    return int(x.data_ptr())


def _is_device(x) -> bool:
    return not isinstance(x, np.ndarray) and getattr(x, "is_cuda", False)


def _i32(seq) -> ctypes.Array | None:
    if seq is None:
        return None
    a = np.ascontiguousarray(np.asarray(seq, dtype=np.int32))
    return (ctypes.c_int32 * max(1, a.size))(*a.tolist())


def _stream(stream) -> int:
    if stream is not None:
        return stream if isinstance(stream, int) else int(stream.cuda_stream)
    import torch
    return int(torch.cuda.current_stream().cuda_stream)


def milo_cache_create(block_tokens: Sequence[int], rank_k: Sequence[int], rank_v: Sequence[int],
                      n_kv_heads: int, head_dim: int, pk, rk, pv, rv, stream=None) -> int:
    """Build a cache from per-block bf16 factors (numpy uint16 arrays in host memory,
    or device tensors); returns the opaque handle as an int."""
    nb = len(pk)
    if not (len(rk) == len(pv) == len(rv) == nb):
        raise ValueError("factor lists differ in length")
    srcs = [pk, rk, pv, rv]
    on_dev = {_is_device(x) for s in srcs for x in s}
    if len(on_dev) > 1:
        raise ValueError("factors must all be host arrays or all device tensors")
    src_on_device = 1 if on_dev == {True} else 0
    keep = []
    arrays = []
    for s in srcs:
        ptrs = (ctypes.c_void_p * nb)()
        for b, x in enumerate(s):
            if isinstance(x, np.ndarray):
                x = np.ascontiguousarray(x, dtype=np.uint16)
                keep.append(x)
            elif not x.is_contiguous():
                raise ValueError("device factors must be contiguous")
            ptrs[b] = _addr(x)
        arrays.append(ptrs)
    bt, rks, rvs = _i32(block_tokens), _i32(rank_k), _i32(rank_v)
    desc = milo_cache_desc(nb, n_kv_heads, head_dim, bt, rks, rvs)
    out = ctypes.c_void_p()
    s = _stream(stream) if src_on_device else (0 if stream is None else _stream(stream))
    _check(lib().milo_cache_create(ctypes.byref(desc), *arrays, src_on_device, s, ctypes.byref(out)))
    return out.value


def milo_attend_decode(cache: int, block_table, q, tail_k, tail_v, tail_len, scale: float, out,
                       stream=None, n_q: int | None = None, n_q_heads: int | None = None,
                       tail_cap: int | None = None) -> None:
    """Queue one decode step.  q: bf16 [n_q][H_q][d], tail_k/v: bf16
    [n_q][tail_cap][H_kv][d], out: fp32 [n_q][H_q][d] (device tensors)."""
    if n_q is None:
        n_q, n_q_heads = int(q.shape[0]), int(q.shape[1])
    if tail_cap is None:
        tail_cap = 0 if tail_k is None else int(tail_k.shape[1])
    table = None if block_table is None else list(block_table)
    n_sel = 0 if table is None else len(table)
    _check(lib().milo_attend_decode(
        ctypes.c_void_p(cache), _i32(table) if n_sel else None, n_sel, n_q, n_q_heads,
        _addr(q), _addr(tail_k), _addr(tail_v), _i32(tail_len), tail_cap, float(scale), _addr(out),
        _stream(stream)))


def milo_attend_prefill(cache: int, block_table, q, tail_k, tail_v, tail_base: int, scale: float, out,
                        stream=None) -> None:
    """Queue the causal prefill of one request's chunk of n_tok tokens.  q: bf16
    [n_tok][H_q][d], tail_k/v: bf16 [tail_cap][H_kv][d] (one shared tail whose rows
    tail_base .. tail_base + n_tok - 1 are the chunk's own keys / values), out: fp32
    [n_tok][H_q][d] (device tensors)."""
    n_tok, n_q_heads = int(q.shape[0]), int(q.shape[1])
    tail_cap = int(tail_k.shape[0])
    table = None if block_table is None else list(block_table)
    n_sel = 0 if table is None else len(table)
    _check(lib().milo_attend_prefill(
        ctypes.c_void_p(cache), _i32(table) if n_sel else None, n_sel, n_tok, n_q_heads,
        _addr(q), _addr(tail_k), _addr(tail_v), int(tail_base), tail_cap, float(scale), _addr(out),
        _stream(stream)))


def milo_allocate_ranks(sigma, n_sv, r_total: int, r_min: int, r_max: int, stream=None) -> np.ndarray:
    """Per-block ranks (Sec. 4.3 allocation).  sigma: device fp32 [n_blocks][ld]
    tensor of non-increasing singular values, n_sv: host [n_blocks] counts.
    Returns int32 [n_blocks]; synchronous."""
    n_blocks, ld = int(sigma.shape[0]), int(sigma.shape[1])
    out = (ctypes.c_int32 * max(1, n_blocks))()
    _check(lib().milo_allocate_ranks(_addr(sigma), ld, n_blocks, _i32(n_sv), int(r_total), int(r_min),
                                     int(r_max), out, _stream(stream)))
    return np.frombuffer(out, dtype=np.int32, count=n_blocks).copy()


def milo_cache_free(cache: int | None) -> None:
    lib().milo_cache_free(ctypes.c_void_p(cache) if cache else None)


def milo_cache_device_bytes(cache: int) -> int:
    v = ctypes.c_int64()
    _check(lib().milo_cache_device_bytes(ctypes.c_void_p(cache), ctypes.byref(v)))
    return v.value


def milo_cache_read_factor(cache: int, block: int, which: int, shape) -> np.ndarray:
    dst = np.zeros(shape, dtype=np.uint16)
    _check(lib().milo_cache_read_factor(ctypes.c_void_p(cache), block, which, dst.ctypes.data))
    return dst


def milo_timing_enable(enable: bool) -> None:
    _check(lib().milo_timing_enable(1 if enable else 0))


def milo_timing_read_alloc():
    """(allocation kernel-chain ms, histogram-pass ms, number of calls) since the last read."""
    a, h, n = ctypes.c_double(), ctypes.c_double(), ctypes.c_int64()
    _check(lib().milo_timing_read_alloc(ctypes.byref(a), ctypes.byref(h), ctypes.byref(n)))
    return a.value, h.value, n.value


def milo_timing_read():
    """(attend-kernel ms, merge-kernel ms, number of calls) since the last read."""
    a, m, n = ctypes.c_double(), ctypes.c_double(), ctypes.c_int64()
    _check(lib().milo_timing_read(ctypes.byref(a), ctypes.byref(m), ctypes.byref(n)))
    return a.value, m.value, n.value
