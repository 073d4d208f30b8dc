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


MILO_P_BF16 = 0
MILO_P_INT8 = 1
MILO_PATH_LATENT = 0
MILO_PATH_RECONSTRUCT = 1
MILO_PATH_AUTO = 2


class milo_cache_desc(ctypes.Structure):
    _fields_ = [("n_blocks", ctypes.c_int32), ("n_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("block_tokens", _c_i32p),
                ("rank_k", _c_i32p), ("rank_v", _c_i32p), ("p_format", ctypes.c_int32)]


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
        L.milo_attend_decode_noalloc.argtypes = [vp, _c_i32p, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                                                 vp, vp, vp, _c_i32p, ctypes.c_int32, ctypes.c_float, vp, vp]
        L.milo_attend_decode_noalloc.restype = ctypes.c_int
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
        L.milo_block_svd.argtypes = [ctypes.POINTER(vp), _c_i32p, ctypes.c_int32, ctypes.c_int32, vp, vp, vp]
        L.milo_block_svd.restype = ctypes.c_int
        L.milo_block_factors.argtypes = [ctypes.POINTER(vp), _c_i32p, ctypes.c_int32, ctypes.c_int32, vp, _c_i32p,
                                         ctypes.POINTER(vp), ctypes.POINTER(vp), vp]
        L.milo_block_factors.restype = ctypes.c_int
        L.milo_block_svd_sweeps.argtypes = [_c_i32p]
        L.milo_block_svd_sweeps.restype = ctypes.c_int
        L.milo_block_svd_flops.argtypes = [ctypes.POINTER(ctypes.c_double)]
        L.milo_block_svd_flops.restype = ctypes.c_int
        L.milo_cache_read_int8.argtypes = [vp, ctypes.c_int32, ctypes.c_int32, vp, vp]
        L.milo_cache_read_int8.restype = ctypes.c_int
        L.milo_cache_plan_builds.argtypes = [vp, ctypes.POINTER(ctypes.c_int64)]
        L.milo_cache_plan_builds.restype = ctypes.c_int
        L.milo_cache_read_factor.argtypes = [vp, ctypes.c_int32, ctypes.c_int32, vp]
        L.milo_cache_read_factor.restype = ctypes.c_int
        L.milo_timing_enable.argtypes = [ctypes.c_int]
        L.milo_timing_enable.restype = ctypes.c_int
        L.milo_timing_read.argtypes = [ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_double),
                                       ctypes.POINTER(ctypes.c_int64)]
        L.milo_timing_read.restype = ctypes.c_int
        L.milo_timing_read_recon.argtypes = [ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_int64)]
        L.milo_timing_read_recon.restype = ctypes.c_int
        L.milo_cache_set_path.argtypes = [vp, ctypes.c_int32]
        L.milo_cache_set_path.restype = ctypes.c_int
        L.milo_cache_recon_blocks.argtypes = [vp, _c_i32p]
        L.milo_cache_recon_blocks.restype = ctypes.c_int
        L.milo_cache_set_rope.argtypes = [vp, ctypes.c_double, ctypes.POINTER(ctypes.c_int64)]
        L.milo_cache_set_rope.restype = ctypes.c_int
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


# shapes of the caches this process created: handle -> (n_blocks, n_kv_heads, head_dim)
_CACHES: dict = {}
_BF16_DTYPES = ("torch.bfloat16", "torch.int16", "torch.uint16")  # bf16 values or their bit patterns


def _dev_tensor(x, name: str, dtypes, ndim: int | None = None):
    """Require a contiguous tensor on the current GPU with one of `dtypes`
    (names), so that no host pointer, wrong element type or strided view ever
    reaches a kernel."""
    import torch
    if not isinstance(x, torch.Tensor):
        raise ValueError(f"{name} must be a torch tensor on the GPU, got {type(x).__name__}")
    if not x.is_cuda:
        raise ValueError(f"{name} must be on the GPU (got device {x.device})")
    if x.device.index != torch.cuda.current_device():
        raise ValueError(f"{name} is on {x.device}, the current device is cuda:{torch.cuda.current_device()}")
    if str(x.dtype) not in dtypes:
        raise ValueError(f"{name} must have dtype {' or '.join(dtypes)}, got {x.dtype}")
    if not x.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if ndim is not None and x.dim() != ndim:
        raise ValueError(f"{name} must have {ndim} dimensions, got shape {tuple(x.shape)}")
    return x


def _is_device(x) -> bool:
    return not isinstance(x, np.ndarray) and getattr(x, "is_cuda", False)


class _I32Arg:
    """An int32 host array passed by pointer (no element-wise copy); keeps the
    numpy buffer alive for the duration of the call."""

    def __init__(self, seq):
        self.a = np.ascontiguousarray(np.asarray(seq, dtype=np.int32).reshape(-1))
        if self.a.size == 0:
            self.a = np.zeros(1, dtype=np.int32)
        self._as_parameter_ = self.a.ctypes.data_as(_c_i32p)


def _i32(seq) -> _I32Arg | None:
    if seq is None:
        return None
    return _I32Arg(seq)


def _stream(stream) -> int:
    if stream is not None:
        return stream if isinstance(stream, int) else int(stream.cuda_stream)
    import torch
    return int(torch.cuda.current_stream().cuda_stream)


def milo_cache_create(block_tokens: Sequence[int], rank_k: Sequence[int], rank_v: Sequence[int],
                      n_kv_heads: int, head_dim: int, pk, rk, pv, rv, stream=None, p_int8: bool = False) -> int:
    """Build a cache from per-block bf16 factors (numpy uint16 arrays in host memory,
    or device tensors); returns the opaque handle as an int.  p_int8 stores P^K and
    P^V as int8 codes with per-token scales (MILO_P_INT8)."""
    nb = len(pk)
    if not (len(rk) == len(pv) == len(rv) == nb):
        raise ValueError("factor lists differ in length")
    srcs = [pk, rk, pv, rv]
    on_dev = {_is_device(x) for s in srcs for x in s}
    if len(on_dev) > 1:
        raise ValueError("factors must all be host arrays or all device tensors")
    src_on_device = 1 if on_dev == {True} else 0
    if not (len(block_tokens) == len(rank_k) == len(rank_v) == nb):
        raise ValueError("block_tokens / rank_k / rank_v must hold one entry per block")
    D = int(n_kv_heads) * int(head_dim)
    keep = []
    arrays = []
    for kind, s in zip(("P^K", "R^K", "P^V", "R^V"), srcs):
        ptrs = (ctypes.c_void_p * nb)()
        for b, x in enumerate(s):
            r = int(rank_k[b] if kind[-1] == "K" else rank_v[b])
            want = (int(block_tokens[b]), r) if kind[0] == "P" else (r, D)
            if tuple(x.shape) != want:
                raise ValueError(f"block {b}: {kind} has shape {tuple(x.shape)}, expected {want}")
            if isinstance(x, np.ndarray):
                if x.dtype not in (np.uint16, np.int16):
                    raise ValueError(f"block {b}: host {kind} must hold bf16 bit patterns (uint16), got {x.dtype}")
                x = np.ascontiguousarray(x).view(np.uint16)
                keep.append(x)
            else:
                _dev_tensor(x, f"block {b} {kind}", _BF16_DTYPES)
            ptrs[b] = _addr(x)
        arrays.append(ptrs)
    bt, rks, rvs = _i32(block_tokens), _i32(rank_k), _i32(rank_v)
    desc = milo_cache_desc(nb, n_kv_heads, head_dim, bt._as_parameter_, rks._as_parameter_, rvs._as_parameter_,
                           MILO_P_INT8 if p_int8 else MILO_P_BF16)
    out = ctypes.c_void_p()
    s = _stream(stream) if src_on_device else (0 if stream is None else _stream(stream))
    _check(lib().milo_cache_create(ctypes.byref(desc), *arrays, src_on_device, s, ctypes.byref(out)))
    _CACHES[out.value] = (nb, int(n_kv_heads), int(head_dim))
    return out.value


def _check_attend_args(cache, q, tail_k, tail_v, out, tail_rank: int):
    """Shapes and element types of an attention call against the cache's
    (n_kv_heads, head_dim); tail_rank is 4 for per-request tails, 3 for one
    shared tail."""
    _dev_tensor(q, "q", _BF16_DTYPES, 3)
    _dev_tensor(out, "out", ("torch.float32",), 3)
    if tuple(out.shape) != tuple(q.shape):
        raise ValueError(f"out shape {tuple(out.shape)} differs from q shape {tuple(q.shape)}")
    shape = _CACHES.get(cache)
    if shape is None:
        raise ValueError("unknown cache handle (not created by milo_cache_create, or already freed)")
    _, n_kv, d = shape
    if q.shape[2] != d:
        raise ValueError(f"q head dim {q.shape[2]} differs from the cache's {d}")
    if tail_k is None and tail_v is None:
        return
    for name, t in (("tail_k", tail_k), ("tail_v", tail_v)):
        if t is None:
            raise ValueError(f"{name} is None while the other tail is given")
        _dev_tensor(t, name, _BF16_DTYPES, tail_rank)
        if tuple(t.shape[-2:]) != (n_kv, d):
            raise ValueError(f"{name} rows must be [H_kv={n_kv}][d={d}], got {tuple(t.shape)}")
    if tuple(tail_k.shape) != tuple(tail_v.shape):
        raise ValueError("tail_k and tail_v differ in shape")
    if tail_rank == 4 and tail_k.shape[0] != q.shape[0]:
        raise ValueError(f"tails hold {tail_k.shape[0]} requests, q holds {q.shape[0]}")


def milo_attend_decode(cache: int, block_table, q, tail_k, tail_v, tail_len, scale: float, out,
                       stream=None, n_q: int | None = None, n_q_heads: int | None = None,
                       tail_cap: int | None = None) -> None:
    """Queue one decode step.  q: bf16 [n_q][H_q][d], tail_k/v: bf16
    [n_q][tail_cap][H_kv][d], out: fp32 [n_q][H_q][d] (device tensors)."""
    _check_attend_args(cache, q, tail_k, tail_v, out, 4)
    if n_q is None:
        n_q, n_q_heads = int(q.shape[0]), int(q.shape[1])
    elif n_q * n_q_heads * q.shape[2] != q.numel():
        raise ValueError(f"n_q={n_q}, n_q_heads={n_q_heads} do not match q of shape {tuple(q.shape)}")
    if tail_cap is None:
        tail_cap = 0 if tail_k is None else int(tail_k.shape[1])
    elif tail_k is not None and tail_cap != tail_k.shape[1]:
        raise ValueError(f"tail_cap={tail_cap} differs from the tails' {tail_k.shape[1]} rows")
    if tail_cap > 0:
        if tail_len is None or len(tail_len) != n_q:
            raise ValueError(f"tail_len must hold {n_q} lengths")
    table = None if block_table is None else np.asarray(block_table, dtype=np.int32).reshape(-1)
    n_sel = 0 if table is None else int(table.size)
    _check(lib().milo_attend_decode(
        ctypes.c_void_p(cache), _i32(table) if n_sel else None, n_sel, n_q, n_q_heads,
        _addr(q), _addr(tail_k), _addr(tail_v), _i32(tail_len), tail_cap, float(scale), _addr(out),
        _stream(stream)))


def milo_attend_decode_noalloc(cache: int, block_table, q, tail_k, tail_v, tail_len, scale: float, out,
                               stream=None) -> None:
    """milo_attend_decode with its workspace in the library's fixed scratch
    (no device allocation; see include/milo.h for the limits)."""
    _check_attend_args(cache, q, tail_k, tail_v, out, 4)
    n_q, n_q_heads = int(q.shape[0]), int(q.shape[1])
    tail_cap = 0 if tail_k is None else int(tail_k.shape[1])
    if tail_cap > 0 and (tail_len is None or len(tail_len) != n_q):
        raise ValueError(f"tail_len must hold {n_q} lengths")
    table = None if block_table is None else np.asarray(block_table, dtype=np.int32).reshape(-1)
    n_sel = 0 if table is None else int(table.size)
    _check(lib().milo_attend_decode_noalloc(
        ctypes.c_void_p(cache), _i32(table) if n_sel else None, n_sel, n_q, n_q_heads,
        _addr(q), _addr(tail_k), _addr(tail_v), _i32(tail_len), tail_cap, float(scale), _addr(out),
        _stream(stream)))


def milo_attend_prefill(cache: int, block_table, q, tail_k, tail_v, tail_base: int, scale: float, out,
                        stream=None) -> None:
    """Queue the causal prefill of one request's chunk of n_tok tokens.  q: bf16
    [n_tok][H_q][d], tail_k/v: bf16 [tail_cap][H_kv][d] (one shared tail whose rows
    tail_base .. tail_base + n_tok - 1 are the chunk's own keys / values), out: fp32
    [n_tok][H_q][d] (device tensors)."""
    _check_attend_args(cache, q, tail_k, tail_v, out, 3)
    if tail_k is None:
        raise ValueError("prefill needs the request's tail (its chunk's own keys and values)")
    n_tok, n_q_heads = int(q.shape[0]), int(q.shape[1])
    tail_cap = int(tail_k.shape[0])
    table = None if block_table is None else np.asarray(block_table, dtype=np.int32).reshape(-1)
    n_sel = 0 if table is None else int(table.size)
    _check(lib().milo_attend_prefill(
        ctypes.c_void_p(cache), _i32(table) if n_sel else None, n_sel, n_tok, n_q_heads,
        _addr(q), _addr(tail_k), _addr(tail_v), int(tail_base), tail_cap, float(scale), _addr(out),
        _stream(stream)))


def milo_allocate_ranks(sigma, n_sv, r_total: int, r_min: int, r_max: int, stream=None) -> np.ndarray:
    """Per-block ranks (Sec. 4.3 allocation).  sigma: device fp32 [n_blocks][ld]
    tensor of non-increasing singular values, n_sv: host [n_blocks] counts.
    Returns int32 [n_blocks]; synchronous."""
    import torch
    if not isinstance(sigma, torch.Tensor) or not sigma.is_cuda or sigma.dtype != torch.float32 \
            or sigma.dim() != 2 or sigma.stride(1) != 1:
        raise ValueError("sigma must be a float32 GPU tensor [n_blocks][ld] with unit column stride")
    if sigma.device.index != torch.cuda.current_device():
        raise ValueError(f"sigma is on {sigma.device}, the current device is cuda:{torch.cuda.current_device()}")
    n_blocks, ld = int(sigma.shape[0]), int(sigma.stride(0)) if sigma.shape[0] > 1 else int(sigma.shape[1])
    if len(n_sv) != n_blocks:
        raise ValueError(f"n_sv must hold {n_blocks} counts")
    if n_blocks > 0 and max(int(v) for v in n_sv) > sigma.shape[1]:
        raise ValueError("a block's singular-value count exceeds the row length")
    out = (ctypes.c_int32 * max(1, n_blocks))()
    _check(lib().milo_allocate_ranks(_addr(sigma), ld, n_blocks, _i32(n_sv), int(r_total), int(r_min),
                                     int(r_max), out, _stream(stream)))
    return np.frombuffer(out, dtype=np.int32, count=n_blocks).copy()


def _dev_ptrs(tensors, name, cols=None):
    ptrs = (ctypes.c_void_p * max(1, len(tensors)))()
    for b, x in enumerate(tensors):
        _dev_tensor(x, f"{name}[{b}]", _BF16_DTYPES, 2)
        if cols is not None and x.shape[1] != cols:
            raise ValueError(f"{name}[{b}] has {x.shape[1]} columns, expected {cols}")
        ptrs[b] = x.data_ptr()
    return ptrs


def milo_block_svd(blocks, stream=None):
    """Encoder (Sec. 4.2 Eq. 3): singular values and right singular vectors of
    every block.  blocks: list of device bf16 tensors [T_b][D] (one shared D).
    Returns (sigma float32 [n_blocks][D], vt float32 [n_blocks][D][D]) on the
    GPU; synchronous."""
    import torch
    if not blocks:
        raise ValueError("no blocks")
    D = int(blocks[0].shape[1])
    ptrs = _dev_ptrs(blocks, "blocks", D)
    dev = blocks[0].device
    sigma = torch.empty((len(blocks), D), dtype=torch.float32, device=dev)
    vt = torch.empty((len(blocks), D, D), dtype=torch.float32, device=dev)
    tokens = [int(x.shape[0]) for x in blocks]
    _check(lib().milo_block_svd(ptrs, _i32(tokens), len(blocks), D, sigma.data_ptr(), vt.data_ptr(),
                                _stream(stream)))
    return sigma, vt


def milo_block_svd_sweeps() -> int:
    v = ctypes.c_int32()
    _check(lib().milo_block_svd_sweeps(ctypes.byref(v)))
    return v.value


def milo_block_svd_flops() -> float:
    v = ctypes.c_double()
    _check(lib().milo_block_svd_flops(ctypes.byref(v)))
    return v.value


def milo_block_factors(blocks, vt, ranks, stream=None):
    """The truncated factors P_b = K_b V_r (bf16 [T_b][r_b]) and R_b = V_r^T
    (bf16 [r_b][D]) of every block, as device int16 tensors of bf16 bits."""
    import torch
    D = int(blocks[0].shape[1])
    ptrs = _dev_ptrs(blocks, "blocks", D)
    if tuple(vt.shape) != (len(blocks), D, D) or vt.dtype != torch.float32 or not vt.is_cuda or \
            not vt.is_contiguous():
        raise ValueError("vt must be the float32 [n_blocks][D][D] GPU tensor milo_block_svd returned")
    ranks = [int(r) for r in ranks]
    if len(ranks) != len(blocks):
        raise ValueError("one rank per block")
    dev = blocks[0].device
    ps = [torch.empty((int(x.shape[0]), r), dtype=torch.int16, device=dev) for x, r in zip(blocks, ranks)]
    rs = [torch.empty((r, D), dtype=torch.int16, device=dev) for r in ranks]
    pp = (ctypes.c_void_p * len(ps))(*[p.data_ptr() for p in ps])
    rp = (ctypes.c_void_p * len(rs))(*[r.data_ptr() for r in rs])
    tokens = [int(x.shape[0]) for x in blocks]
    _check(lib().milo_block_factors(ptrs, _i32(tokens), len(blocks), D, vt.data_ptr(), _i32(ranks), pp, rp,
                                    _stream(stream)))
    return ps, rs


def milo_cache_free(cache: int | None) -> None:
    _CACHES.pop(cache, None)
    lib().milo_cache_free(ctypes.c_void_p(cache) if cache else None)


def milo_cache_device_bytes(cache: int) -> int:
    v = ctypes.c_int64()
    _check(lib().milo_cache_device_bytes(ctypes.c_void_p(cache), ctypes.byref(v)))
    return v.value


def milo_cache_read_int8(cache: int, block: int, which: int, shape):
    """INT8 P factors: (codes int8 [T][rank], scales float32 [T]) of P^K (which=0) or P^V (2)."""
    codes = np.zeros(shape, dtype=np.int8)
    scales = np.zeros(shape[0], dtype=np.float32)
    _check(lib().milo_cache_read_int8(ctypes.c_void_p(cache), block, which, codes.ctypes.data, scales.ctypes.data))
    return codes, scales


def milo_cache_set_path(cache: int, path: int) -> None:
    """MILO_PATH_LATENT, MILO_PATH_RECONSTRUCT or MILO_PATH_AUTO (Sec. 4.5 inference path)."""
    _check(lib().milo_cache_set_path(ctypes.c_void_p(cache), int(path)))


def milo_cache_set_rope(cache: int, theta: float, block_pos: Sequence[int] | None = None) -> None:
    """Pre-RoPE keys (Sec. 3): block b's token t sits at block_pos[b] + t (None: the
    blocks one after another in id order); theta = 0 turns the rotation off."""
    pos = None
    if block_pos is not None:
        arr = np.ascontiguousarray(np.asarray(block_pos, dtype=np.int64))
        shape = _CACHES.get(cache)
        if arr.ndim != 1 or (shape is not None and arr.shape[0] != shape[0]):
            raise ValueError(f"block_pos must hold one position per block (got shape {arr.shape})")
        pos = arr.ctypes.data_as(ctypes.POINTER(ctypes.c_int64))
    _check(lib().milo_cache_set_rope(ctypes.c_void_p(cache), float(theta), pos))


def milo_cache_recon_blocks(cache: int) -> int:
    """Blocks the plan of the cache's last attention call reconstructs."""
    v = ctypes.c_int32()
    _check(lib().milo_cache_recon_blocks(ctypes.c_void_p(cache), ctypes.byref(v)))
    return v.value


def milo_timing_read_recon():
    """(reconstruction kernel ms, number of calls) since the last read."""
    t, n = ctypes.c_double(), ctypes.c_int64()
    _check(lib().milo_timing_read_recon(ctypes.byref(t), ctypes.byref(n)))
    return t.value, n.value


def milo_cache_plan_builds(cache: int) -> int:
    """Work plans built for this cache so far."""
    v = ctypes.c_int64()
    _check(lib().milo_cache_plan_builds(ctypes.c_void_p(cache), ctypes.byref(v)))
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
