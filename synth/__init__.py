"""Seeded synthetic inputs for low-rank decode attention.

This module only draws numbers and stores them; it performs none of the
attention arithmetic.  Both the CPU oracle tests and the GPU path consume
what it produces, so it is the one piece of code the two sides share.

Inputs follow the problem statement of block-wise low-rank KV compression
(Sec. 4.2, Eq. 3): every context block b of T_b tokens carries key and value
factors K_b ~ P^K_b R^K_b, V_b ~ P^V_b R^V_b with the singular values already
folded into P, a per-block rank (Sec. 4.3), and one shared rank space across
the KV heads (R has H_kv*d columns, head-major: column g*d + j).  The query's
own uncompressed KV (the "dense tail", Alg. 1 inference stage) is per request.

Random streams: numpy's Philox counter-based generator, one independent key
per (config, layer, tensor, block).  Normals are drawn in fp32 and rounded to
bf16 with round-to-nearest-even.
"""
from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, field

import numpy as np

__all__ = [
    "Config", "CONFIGS", "LayerInputs", "f32_to_bf16", "bf16_to_f32",
    "bf16_to_f64", "gen_layer", "make_problem", "draw_block_tokens",
    "draw_ranks", "algorithmic_bytes", "latent_flops", "recon_flops", "gen_spectra", "Spectra", "gen_kv_block",
]

_MAGIC = 0x4D494C4F  # "MILO"
# tensor ids inside one layer's key space
T_META, T_PK, T_RK, T_PV, T_RV, T_TAILK, T_TAILV, T_Q, T_SIGMA = range(9)
_SHARED_LAYER = 0xFFFFF  # key slot for draws shared by every layer


# --------------------------------------------------------------------------
# bf16 storage helpers (IEEE binary32 truncated to its top 16 bits)
# --------------------------------------------------------------------------
def f32_to_bf16(x: np.ndarray) -> np.ndarray:
    """fp32 -> bf16 bit patterns (uint16), round to nearest, ties to even."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    bias = ((u >> 16) & 1) + np.uint32(0x7FFF)
    return ((u + bias) >> 16).astype(np.uint16)


def bf16_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def bf16_to_f64(b: np.ndarray) -> np.ndarray:
    return bf16_to_f32(b).astype(np.float64)


def _rng(cfg_id: int, layer: int, tensor: int, block: int = 0) -> np.random.Generator:
    k0 = (_MAGIC << 32) | (cfg_id & 0xFFFFFFFF)
    k1 = ((layer & 0xFFFFFF) << 40) | ((tensor & 0xFF) << 32) | (block & 0xFFFFFFFF)
    return np.random.Generator(np.random.Philox(key=np.array([k0, k1], dtype=np.uint64)))


def _normal_bf16(rng: np.random.Generator, shape, std: float = 1.0) -> np.ndarray:
    x = rng.standard_normal(shape, dtype=np.float32)
    if std != 1.0:
        x *= np.float32(std)
    return f32_to_bf16(x)


# --------------------------------------------------------------------------
# Workload configurations (Qwen2.5-shaped single decode steps)
# --------------------------------------------------------------------------
@dataclass(frozen=True)
class Config:
    name: str
    cfg_id: int
    n_layers: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    n_q: int            # decode batch: independent query tokens sharing the context
    tail: int           # dense tail tokens per request
    n_blocks: int       # 0 -> ragged block sizes drawn to sum to `context`
    block_tokens: int   # T_b when uniform
    context: int        # total compressed context tokens C
    rank_rule: str      # see draw_ranks
    description: str = ""

    @property
    def d_kv(self) -> int:
        return self.n_kv_heads * self.head_dim

    @property
    def group(self) -> int:
        return self.n_q_heads // self.n_kv_heads


CONFIGS = {
    "tiny": Config("tiny", 0, 1, 14, 2, 64, 1, 64, 8, 512, 4096, "tiny",
                   "1 layer, 14/2 heads, d=64, 8x512 tokens, r in {32,64,96,128}, tail 64, 1 query"),
    "q7b_1l": Config("q7b_1l", 1, 1, 28, 4, 128, 8, 256, 64, 1024, 65536, "q7b_1l",
                     "Qwen2.5-7B-shaped layer, 64x1024 tokens, r in 64..512 step 32, tail 256, 8 queries"),
    "q7b_28l": Config("q7b_28l", 2, 28, 28, 4, 128, 32, 512, 128, 1024, 131072, "q7b_skewed",
                      "Qwen2.5-7B-shaped, 28 layers, 128x1024 tokens, skewed ranks, tail 512, 32 queries"),
    "q14b_48l": Config("q14b_48l", 3, 48, 40, 8, 128, 64, 1024, 256, 1024, 262144, "q14b",
                       "Qwen2.5-14B-shaped, 48 layers, 256x1024 tokens, r in 128..768 step 64, tail 1024, 64 queries"),
    "q32b_64l": Config("q32b_64l", 4, 64, 40, 8, 128, 16, 2048, 0, 0, 1048576, "q32b",
                       "Qwen2.5-32B-shaped, 64 layers, 1M tokens in ragged {512,1024,2048} blocks, "
                       "r in 128..512 step 32, tail 2048, 16 queries"),
}


def draw_block_tokens(cfg: Config) -> np.ndarray:
    """Block sizes T_b. Uniform configs are fixed; the ragged one draws T_b from
    {512,1024,2048} in sequence until the total is exactly cfg.context (a draw
    that would overshoot is replaced by a draw among the values that fit)."""
    if cfg.n_blocks > 0:
        return np.full(cfg.n_blocks, cfg.block_tokens, dtype=np.int32)
    rng = _rng(cfg.cfg_id, _SHARED_LAYER, T_META)
    choices = np.array([512, 1024, 2048])
    out, left = [], cfg.context
    while left > 0:
        fit = choices[choices <= left]
        t = int(fit[rng.integers(len(fit))])
        out.append(t)
        left -= t
    return np.array(out, dtype=np.int32)


def draw_ranks(cfg: Config, layer: int, n_blocks: int) -> np.ndarray:
    """Per-block rank r_b (used for both K and V), drawn per layer."""
    rng = _rng(cfg.cfg_id, layer, T_META)
    rule = cfg.rank_rule
    if rule == "tiny":
        vals = np.array([32, 64, 96, 128])
        return vals[rng.integers(len(vals), size=n_blocks)].astype(np.int32)
    if rule == "q7b_1l":
        vals = np.arange(64, 513, 32)
        return vals[rng.integers(len(vals), size=n_blocks)].astype(np.int32)
    if rule == "q7b_skewed":
        n_hi = int(round(0.2 * n_blocks))
        hi_idx = rng.permutation(n_blocks)[:n_hi]
        lo_vals, hi_vals = np.array([64, 96, 128, 160]), np.arange(384, 513, 32)
        r = lo_vals[rng.integers(len(lo_vals), size=n_blocks)]
        r[hi_idx] = hi_vals[rng.integers(len(hi_vals), size=n_hi)]
        return r.astype(np.int32)
    if rule == "q14b":
        vals = np.arange(128, 769, 64)
        return vals[rng.integers(len(vals), size=n_blocks)].astype(np.int32)
    if rule == "q32b":
        vals = np.arange(128, 513, 32)
        return vals[rng.integers(len(vals), size=n_blocks)].astype(np.int32)
    raise ValueError(rule)


@dataclass
class LayerInputs:
    """One layer's worth of bf16 inputs (uint16 bit patterns, C-contiguous)."""
    n_kv_heads: int
    head_dim: int
    n_q_heads: int
    block_tokens: np.ndarray          # int32 [nb]
    rank_k: np.ndarray                # int32 [nb]
    rank_v: np.ndarray                # int32 [nb]
    pk: list                          # [nb] uint16 [T_b][rk_b]
    rk: list                          # [nb] uint16 [rk_b][H_kv*d]
    pv: list                          # [nb] uint16 [T_b][rv_b]
    rv: list                          # [nb] uint16 [rv_b][H_kv*d]
    q: np.ndarray                     # uint16 [n_q][H_q][d]
    tail_k: np.ndarray                # uint16 [n_q][tail_cap][H_kv][d]
    tail_v: np.ndarray                # uint16 [n_q][tail_cap][H_kv][d]
    tail_len: np.ndarray              # int32 [n_q]
    scale: float
    meta: dict = field(default_factory=dict)

    @property
    def n_blocks(self) -> int:
        return len(self.pk)

    @property
    def n_q(self) -> int:
        return self.q.shape[0]

    @property
    def tail_cap(self) -> int:
        return self.tail_k.shape[1]


def _workers() -> int:
    return max(1, min(16, os.cpu_count() or 1))


def _gen_factors(cfg_id, layer, T, rk, rv, D, block):
    g1 = _rng(cfg_id, layer, T_PK, block)
    g2 = _rng(cfg_id, layer, T_RK, block)
    g3 = _rng(cfg_id, layer, T_PV, block)
    g4 = _rng(cfg_id, layer, T_RV, block)
    return (_normal_bf16(g1, (T, rk)), _normal_bf16(g2, (rk, D), 1.0 / np.sqrt(rk)),
            _normal_bf16(g3, (T, rv)), _normal_bf16(g4, (rv, D), 1.0 / np.sqrt(rv)))


def _assemble(cfg_id, layer, block_tokens, rank_k, rank_v, n_kv_heads, head_dim, n_q,
              n_q_heads, tail_cap, tail_len, meta) -> LayerInputs:
    D = n_kv_heads * head_dim
    nb = len(block_tokens)
    with ThreadPoolExecutor(_workers()) as ex:
        facs = list(ex.map(lambda b: _gen_factors(cfg_id, layer, int(block_tokens[b]), int(rank_k[b]),
                                                  int(rank_v[b]), D, b), range(nb)))
        tk = ex.submit(lambda: np.stack([_normal_bf16(_rng(cfg_id, layer, T_TAILK, i),
                                                      (tail_cap, n_kv_heads, head_dim))
                                         for i in range(n_q)]) if n_q else None)
        tv = ex.submit(lambda: np.stack([_normal_bf16(_rng(cfg_id, layer, T_TAILV, i),
                                                      (tail_cap, n_kv_heads, head_dim))
                                         for i in range(n_q)]) if n_q else None)
        tail_k, tail_v = tk.result(), tv.result()
    q = _normal_bf16(_rng(cfg_id, layer, T_Q), (n_q, n_q_heads, head_dim))
    return LayerInputs(
        n_kv_heads=n_kv_heads, head_dim=head_dim, n_q_heads=n_q_heads,
        block_tokens=np.asarray(block_tokens, dtype=np.int32),
        rank_k=np.asarray(rank_k, dtype=np.int32), rank_v=np.asarray(rank_v, dtype=np.int32),
        pk=[f[0] for f in facs], rk=[f[1] for f in facs],
        pv=[f[2] for f in facs], rv=[f[3] for f in facs],
        q=q, tail_k=tail_k, tail_v=tail_v,
        tail_len=np.asarray(tail_len, dtype=np.int32),
        scale=float(1.0 / np.sqrt(head_dim)), meta=meta)


def gen_layer(cfg: Config | str, layer: int = 0) -> LayerInputs:
    """All inputs of one layer of a named workload, seeded by (config, layer).
    P ~ N(0,1), R ~ N(0, 1/r_b) (variance), tail K/V ~ N(0,1), q ~ N(0,1)."""
    if isinstance(cfg, str):
        cfg = CONFIGS[cfg]
    bt = draw_block_tokens(cfg)
    r = draw_ranks(cfg, layer, len(bt))
    return _assemble(cfg.cfg_id, layer, bt, r, r, cfg.n_kv_heads, cfg.head_dim, cfg.n_q,
                     cfg.n_q_heads, cfg.tail, np.full(cfg.n_q, cfg.tail, dtype=np.int32),
                     {"config": cfg.name, "layer": layer})


def make_problem(seed: int, block_tokens, rank_k, rank_v=None, *, n_kv_heads=2, head_dim=64,
                 n_q=1, n_q_heads=4, tail_cap=0, tail_len=None) -> LayerInputs:
    """Arbitrary-shape problem for tests (same distributions, own key space)."""
    rank_v = rank_k if rank_v is None else rank_v
    if tail_len is None:
        tail_len = [tail_cap] * n_q
    return _assemble(1000 + seed, 0, list(block_tokens), list(rank_k), list(rank_v), n_kv_heads,
                     head_dim, n_q, n_q_heads, tail_cap, tail_len, {"seed": seed})


# --------------------------------------------------------------------------
# Accounting (what one decode step over one layer must move / compute)
# --------------------------------------------------------------------------
def algorithmic_bytes(inp: LayerInputs, table=None, p_int8: bool = False) -> int:
    """Bytes a step must touch once: every selected factor (bf16; with INT8 P
    factors one byte per P element plus two fp32 scales per token), each
    request's valid tail K/V (bf16), the queries (bf16) and the fp32 output."""
    table = range(inp.n_blocks) if table is None else table
    D = inp.n_kv_heads * inp.head_dim
    if p_int8:
        fac = sum((int(inp.block_tokens[b]) + 2 * D) * (int(inp.rank_k[b]) + int(inp.rank_v[b]))
                  + 8 * int(inp.block_tokens[b]) for b in table)
    else:
        fac = sum(2 * (int(inp.block_tokens[b]) + D) * (int(inp.rank_k[b]) + int(inp.rank_v[b]))
                  for b in table)
    tail = 2 * 2 * int(np.sum(inp.tail_len)) * D
    ncol = inp.n_q * inp.n_q_heads
    return fac + tail + 2 * ncol * inp.head_dim + 4 * ncol * inp.head_dim


def latent_flops(inp: LayerInputs, table=None) -> int:
    """Multiply-add flops of the latent route (projection, scores, latent V,
    up-projection, tail)."""
    table = range(inp.n_blocks) if table is None else table
    ncol = inp.n_q * inp.n_q_heads
    d = inp.head_dim
    blk = sum(2 * ncol * (int(inp.rank_k[b]) + int(inp.rank_v[b])) * (int(inp.block_tokens[b]) + d)
              for b in table)
    G = inp.n_q_heads // inp.n_kv_heads
    tail = 4 * int(np.sum(inp.tail_len)) * G * inp.n_kv_heads * d
    return blk + tail


def recon_flops(inp: LayerInputs, table=None) -> int:
    """Multiply-add flops of the reconstruct-then-attend route with every block
    rebuilt: K_b = P^K R^K and V_b = P^V R^V (2 T D r each), then dense scores
    and value pass (4 N T d), and the tail."""
    table = range(inp.n_blocks) if table is None else table
    ncol = inp.n_q * inp.n_q_heads
    d = inp.head_dim
    D = inp.n_kv_heads * d
    blk = sum(2 * int(inp.block_tokens[b]) * D * (int(inp.rank_k[b]) + int(inp.rank_v[b])) +
              4 * ncol * int(inp.block_tokens[b]) * d for b in table)
    G = inp.n_q_heads // inp.n_kv_heads
    tail = 4 * int(np.sum(inp.tail_len)) * G * inp.n_kv_heads * d
    return blk + tail


# --------------------------------------------------------------------------
# Singular-value spectra for the rank allocation (encoder input)
# --------------------------------------------------------------------------
@dataclass
class Spectra:
    """Per-block singular values of one layer's keys (or values), fp32, each row
    non-increasing; row b holds n_sv[b] = min(T_b, D) values, padded with zeros
    to ld columns; plus the allocation's budget and bounds."""
    sigma: np.ndarray       # float32 [n_blocks][ld]
    n_sv: np.ndarray        # int32 [n_blocks]
    r_total: int
    r_min: int
    r_max: int


def gen_spectra(cfg: Config | str, layer: int = 0, rho: float = 0.5, r_min: int = 32,
                r_max: int = 896) -> Spectra:
    """Seeded synthetic spectra with the block structure of a workload: block b
    decays as a power law sigma_j = s_b (j + 1)^(-a_b) with a_b ~ U(0.2, 1.6) and
    s_b ~ LogNormal(0, 0.5), so blocks range from flat (information-dense) to
    steep (redundant).  About one value in 64 is copied from its predecessor, so
    equal values (ties) occur inside rows.  The budget is the rank sum at which
    Eq. 4's ratio equals rho when every block has the same rank:
    r_total = floor(rho * N * D * B / (B + D)) with B the mean block size."""
    if isinstance(cfg, str):
        cfg = CONFIGS[cfg]
    T = draw_block_tokens(cfg)
    D = cfg.d_kv
    n_sv = np.minimum(T, D).astype(np.int32)
    ld = int(n_sv.max())
    rng = _rng(cfg.cfg_id, layer, T_SIGMA)
    a = rng.uniform(0.2, 1.6, size=len(T))
    s0 = np.exp(rng.normal(0.0, 0.5, size=len(T)))
    sigma = np.zeros((len(T), ld), dtype=np.float32)
    for b, n in enumerate(n_sv):
        row = (s0[b] * np.arange(1, n + 1, dtype=np.float64) ** -a[b]).astype(np.float32)
        dup = np.flatnonzero(rng.random(n) < 1.0 / 64)
        dup = dup[dup > 0]
        row[dup] = row[dup - 1]
        sigma[b, :n] = np.minimum.accumulate(row)
    B = float(T.mean())
    r_total = int(np.floor(rho * len(T) * D * B / (B + D)))
    return Spectra(sigma, n_sv, r_total, r_min, r_max)


# --------------------------------------------------------------------------
# Uncompressed key / value blocks for the encoder (input of the per-block SVD)
# --------------------------------------------------------------------------
def gen_kv_block(seed: int, T: int, D: int, decay: float = 0.8, scale: float = 8.0) -> np.ndarray:
    """A T x D block of keys (or values) with a power-law spectrum:
    K = U diag(sigma) V^T with U, V random orthonormal (QR of Gaussian
    matrices, seeded) and sigma_j = scale (j + 1)^(-decay), j < min(T, D),
    rounded to bf16 (uint16 bit patterns).  Real key blocks are strongly
    low-rank (Sec. 3); the decay sets how much."""
    rng = np.random.Generator(np.random.Philox(key=[_MAGIC, 0x5356 + seed]))
    n = min(T, D)
    u, _ = np.linalg.qr(rng.standard_normal((T, n)))
    v, _ = np.linalg.qr(rng.standard_normal((D, n)))
    sig = scale * np.arange(1, n + 1, dtype=np.float64) ** -decay
    return f32_to_bf16(((u * sig) @ v.T).astype(np.float32))
