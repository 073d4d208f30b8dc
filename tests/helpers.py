"""Shared test plumbing: turn bf16 synthetic inputs into the oracle's fp64
arguments, run the GPU path through the C ABI, and measure the per-column
relative L2 error used as the parity bar."""
import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

from synth import LayerInputs, bf16_to_f64

TOL_REL_L2 = 1e-2   # max over (query, head) of ||o_gpu - o_ref|| / ||o_ref||


def _conv_list(xs):
    with ThreadPoolExecutor(max(1, min(16, os.cpu_count() or 1))) as ex:
        return list(ex.map(bf16_to_f64, xs))


def oracle_args(inp: LayerInputs, table=None, tail_len=None):
    return dict(
        pk=_conv_list(inp.pk), rk=_conv_list(inp.rk), pv=_conv_list(inp.pv), rv=_conv_list(inp.rv),
        table=list(range(inp.n_blocks)) if table is None else list(table),
        q=bf16_to_f64(inp.q), tail_k=bf16_to_f64(inp.tail_k), tail_v=bf16_to_f64(inp.tail_v),
        tail_len=inp.tail_len if tail_len is None else np.asarray(tail_len), scale=inp.scale)


def oracle_args_int8(inp: LayerInputs, table=None, tail_len=None):
    """The oracle's arguments for a cache that stores P^K and P^V as INT8: the
    dequantised P factors (oracle.quantize_rows_int8 of the bf16 values), the
    bf16 R factors, queries and tails."""
    import oracle
    from synth import bf16_to_f32
    a = oracle_args(inp, table, tail_len)
    deq = lambda x: oracle.dequantize_rows_int8(*oracle.quantize_rows_int8(bf16_to_f32(x)))
    with ThreadPoolExecutor(max(1, min(16, os.cpu_count() or 1))) as ex:
        a["pk"] = list(ex.map(deq, inp.pk))
        a["pv"] = list(ex.map(deq, inp.pv))
    return a


def col_rel_l2(got: np.ndarray, ref: np.ndarray) -> np.ndarray:
    d = ref.shape[-1]
    got = np.asarray(got, dtype=np.float64).reshape(-1, d)
    ref = np.asarray(ref, dtype=np.float64).reshape(-1, d)
    return np.linalg.norm(got - ref, axis=1) / np.maximum(np.linalg.norm(ref, axis=1), 1e-300)


def max_rel_l2(got: np.ndarray, ref: np.ndarray) -> float:
    """max over (query, head) columns of ||got - ref||_2 / ||ref||_2."""
    return float(np.max(col_rel_l2(got, ref)))


# ------------------------------------------------------------------------------
# GPU side (only through the C ABI)
# ------------------------------------------------------------------------------
def to_device(a: np.ndarray):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).cuda()


class GpuLayer:
    """A cache built from one LayerInputs plus device copies of q and the tails."""

    def __init__(self, inp: LayerInputs, src_on_device=False, p_int8=False):
        from paper_2609_29913_amd import milo
        self.inp = inp
        if src_on_device:
            facs = [[to_device(x) for x in lst] for lst in (inp.pk, inp.rk, inp.pv, inp.rv)]
        else:
            facs = [inp.pk, inp.rk, inp.pv, inp.rv]
        self.cache = milo.milo_cache_create(inp.block_tokens, inp.rank_k, inp.rank_v, inp.n_kv_heads,
                                            inp.head_dim, *facs, p_int8=p_int8)
        self.q = to_device(inp.q)
        self.tk = to_device(inp.tail_k)
        self.tv = to_device(inp.tail_v)

    def attend(self, table=None, tail_len=None, out=None, fill=float("nan")):
        import torch
        from paper_2609_29913_amd import milo
        inp = self.inp
        table = list(range(inp.n_blocks)) if table is None else list(table)
        tail_len = inp.tail_len if tail_len is None else tail_len
        if out is None:
            out = torch.full(inp.q.shape, fill, dtype=torch.float32, device="cuda")
        milo.milo_attend_decode(self.cache, table, self.q, self.tk, self.tv, tail_len, inp.scale, out)
        torch.cuda.synchronize()
        return out

    def free(self):
        from paper_2609_29913_amd import milo
        milo.milo_cache_free(self.cache)
        self.cache = None
