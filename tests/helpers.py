"""Shared test plumbing: turn bf16 synthetic inputs into the oracle's fp64 arguments
and measure the per-column relative L2 error used as the parity bar."""
import numpy as np

from synth import LayerInputs, bf16_to_f64


def oracle_args(inp: LayerInputs, table=None, tail_len=None):
    return dict(
        pk=[bf16_to_f64(x) for x in inp.pk], rk=[bf16_to_f64(x) for x in inp.rk],
        pv=[bf16_to_f64(x) for x in inp.pv], rv=[bf16_to_f64(x) for x in inp.rv],
        table=list(range(inp.n_blocks)) if table is None else list(table),
        q=bf16_to_f64(inp.q), tail_k=bf16_to_f64(inp.tail_k), tail_v=bf16_to_f64(inp.tail_v),
        tail_len=inp.tail_len if tail_len is None else np.asarray(tail_len), scale=inp.scale)


def max_rel_l2(got: np.ndarray, ref: np.ndarray) -> float:
    """max over (query, head) columns of ||got - ref||_2 / ||ref||_2."""
    got = np.asarray(got, dtype=np.float64).reshape(-1, ref.shape[-1])
    ref = np.asarray(ref, dtype=np.float64).reshape(-1, ref.shape[-1])
    num = np.linalg.norm(got - ref, axis=1)
    den = np.linalg.norm(ref, axis=1)
    return float(np.max(num / np.maximum(den, 1e-300)))
