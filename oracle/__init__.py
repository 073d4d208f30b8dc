"""CPU oracle for decode attention over a block-wise low-rank KV cache.

TEST INFRASTRUCTURE ONLY.  Nothing on the product path may import, call or
execute this package: only the tests, the package smoke check and the
benchmark's CPU-baseline leg use it.  It shares no code with the GPU library
and imports nothing from it; it takes plain float64 arrays.

What it computes (the method's result, written out plainly in fp64):

* Each context block b is stored as factors of its keys and values
  (Sec. 4.2, Eq. 3), with the diagonal of singular values already multiplied
  into the left factor:  K_b = P^K_b R^K_b,  V_b = P^V_b R^V_b.
  P^*_b is T_b x r_b, R^*_b is r_b x (H_kv*d); the columns of R are head-major,
  so KV head g owns columns g*d .. g*d+d-1.
* At inference the selected blocks (Alg. 1 inference stage; the caller's block
  table stands in for the retriever) and the request's own uncompressed KV are
  attended together with scaled dot-product attention (Sec. 4.1, Eq. 1).
* Query head h reads KV head g = floor(h / G), G = H_q / H_kv.

`attend_dense` is that definition: rebuild K and V, then softmax attention.
`attend_prefill` is the same definition for a multi-token input query of one
request whose tokens attend causally among themselves (a chunk of new tokens
sharing one tail).
`quantize_rows_int8` is the INT8 storage of a P factor (Sec. 5.3 combines the
low-rank cache with INT8 quantisation): one scale per token row.
`block_svd` / `block_factors` are the encoder's per-block truncated SVD (Sec.
4.2 Eq. 3, Alg. 1 encoding stage): the singular values and right singular
vectors of a block's keys (or values), then P = U_r Sigma_r = K V_r, R = V_r^T.
`allocate_ranks` is the encoder's rank allocation (Sec. 4.3): per-block ranks
that maximise the retained spectral information (Eq. 5) under a total rank
budget and per-block bounds (Eq. 6), found by the greedy over marginal gains
(Eq. 7) that the paper describes.

`rope` is the rotary position embedding of the Qwen2 models the paper
measures (Sec. 3 studies, and Sec. 4.2 factorises, the keys before it is
applied); `attend_dense` and `attend_prefill` apply it to the keys that the
factors define when they are given the blocks' positions, which is what
attending such a cache by reconstruction means (Sec. 4.5, Alg. 1 full-rank
reconstruction: the rank space cannot carry the rotation).

`attend_latent` reaches the same numbers by exact reassociation,
q.(P R)_t = P_t.(R q) and sum_t w_t (P R)_t = (sum_t w_t P_t) R, which is the
order the GPU path follows: project the query per block, score against P^K
rows, softmax over all keys, accumulate weights times P^V rows in rank space,
up-project through R^V, add the dense tail, normalise.  Both use one global
maximum per column (two-pass softmax) and sum blocks in table order, tokens
ascending, then the tail.
"""
from __future__ import annotations

import math

import numpy as np

__all__ = ["allocate_ranks", "attend_dense", "attend_latent", "attend_prefill", "block_factors", "block_svd",
           "dequantize_rows_int8", "quantize_rows_int8", "reconstruct", "rope", "spectral_information"]


def _mm(a: np.ndarray, b: np.ndarray, ordered: bool) -> np.ndarray:
    """a @ b for a 2-D a and a 1-D or 2-D b.  With ordered=True the sum over the
    shared index runs strictly left to right (one rounded product and one rounded
    addition per term, starting from 0), so the result does not depend on how a
    library blocks the sum; otherwise BLAS."""
    if not ordered:
        return a @ b
    out = np.zeros((a.shape[0],) + b.shape[1:], dtype=np.result_type(a, b))
    for k in range(a.shape[1]):
        out += np.multiply.outer(a[:, k], b[k])
    return out


def _colsum(w: np.ndarray, ordered: bool):
    """Sum over the first axis (tokens); left to right when ordered."""
    if not ordered:
        return w.sum(axis=0)
    out = np.zeros(w.shape[1:], dtype=w.dtype)
    for t in range(w.shape[0]):
        out += w[t]
    return out


def _exp(x: np.ndarray, ordered: bool) -> np.ndarray:
    """Elementwise exp; with ordered=True one math.exp call per element, so two
    arrays holding the same value get the same result whatever their shapes."""
    if not ordered:
        return np.exp(x)
    return np.vectorize(math.exp, otypes=[np.float64])(x) if x.size else np.exp(x)


def reconstruct(p: np.ndarray, r: np.ndarray, ordered: bool = False) -> np.ndarray:
    """Eq. 3 with the singular values folded into P: the dense block P R."""
    return _mm(p, r, ordered)


def rope(x, positions, theta: float) -> np.ndarray:
    """Rotary position embedding (RoFormer, Su et al.) in the rotate-half
    arrangement of the Qwen2 models the paper measures.  Along the last axis
    (length d, even), element j < d/2 pairs with element j + d/2; the pair (u, v)
    of a row at position p turns by the angle p * theta^(-2j/d):
        (u, v) -> (u cos - v sin,  v cos + u sin).
    positions holds one integer per index of the first axis; the angles are
    formed in float64 from the integer position.  Returns a new float64 array."""
    x = np.asarray(x, dtype=np.float64)
    d = x.shape[-1]
    if d % 2:
        raise ValueError("the rotated axis must have even length")
    pos = np.asarray(positions, dtype=np.int64)
    if pos.shape != x.shape[:1]:
        raise ValueError("one position per row of the first axis")
    freq = float(theta) ** (-2.0 * np.arange(d // 2, dtype=np.float64) / d)
    ang = pos.astype(np.float64)[:, None] * freq[None, :]       # [rows, d/2]
    ang = ang.reshape(ang.shape[:1] + (1,) * (x.ndim - 2) + ang.shape[1:])
    c, s = np.cos(ang), np.sin(ang)
    u, v = x[..., : d // 2], x[..., d // 2:]
    return np.concatenate([u * c - v * s, v * c + u * s], axis=-1)


def _block_keys(pk, rk, b, d, key_pos, rope_theta, ordered):
    """The keys block b's factors define (Eq. 3), rotated to the block's
    positions key_pos[b] + t when key_pos is given (pre-RoPE keys)."""
    k = reconstruct(pk[b], rk[b], ordered)
    if key_pos is None:
        return k
    T = k.shape[0]
    kh = k.reshape(T, -1, d)                               # [T, H_kv, d]
    return rope(kh, int(key_pos[b]) + np.arange(T), rope_theta).reshape(T, -1)


def _shapes(q, rk_list, tail_k):
    n_q, n_q_heads, d = q.shape
    n_kv = tail_k.shape[2]
    if n_q_heads % n_kv:
        raise ValueError("query heads must be a multiple of KV heads")
    for r in rk_list:
        if r.shape[1] != n_kv * d:
            raise ValueError("R must have H_kv*d columns")
    return n_q, n_q_heads, d, n_kv, n_q_heads // n_kv


def attend_dense(pk, rk, pv, rv, table, q, tail_k, tail_v, tail_len, scale, ordered=False, key_pos=None,
                 rope_theta=None):
    """Definition: Eq. 1 over the keys/values that the factors of the selected
    blocks define (Eq. 3), in table order, followed by request i's first
    tail_len[i] uncompressed tail tokens:
        o = sum_t e^{s_t - M} v_t / sum_t e^{s_t - M},  s_t = scale q . k_t,  M = max_t s_t,
    both sums taken block by block (tokens ascending) in table order, then over
    the tail.  ordered=True makes every dot product and sum run left to right
    (see _mm), which fixes the result to the last bit.

    pk, rk, pv, rv: lists (indexed by block id) of float64 arrays
        P^K_b [T_b, rk_b], R^K_b [rk_b, H_kv*d], P^V_b [T_b, rv_b], R^V_b [rv_b, H_kv*d]
    table: selected block ids, in order
    q: [n_q, H_q, d]; tail_k, tail_v: [n_q, tail_cap, H_kv, d]; tail_len: [n_q]
    key_pos, rope_theta: optional (pre-RoPE keys): key_pos indexed by block id
        gives the position of the block's first token; the key of token t is
        then rope(K_b[t], key_pos[b] + t, rope_theta), per KV head.  The
        queries and the tail keys are taken as already rotated.
    returns o: [n_q, H_q, d] float64
    """
    n_q, n_q_heads, d, n_kv, G = _shapes(q, [rk[b] for b in table], tail_k)
    keys = [_block_keys(pk, rk, b, d, key_pos, rope_theta, ordered) for b in table]
    vals = [reconstruct(pv[b], rv[b], ordered) for b in table]
    out = np.empty((n_q, n_q_heads, d))
    for i in range(n_q):
        n_t = int(tail_len[i])
        for h in range(n_q_heads):
            g = h // G
            cols = slice(g * d, (g + 1) * d)       # KV head g's columns of K and V
            k_parts = [k[:, cols] for k in keys] + [tail_k[i, :n_t, g, :]]
            v_parts = [v[:, cols] for v in vals] + [tail_v[i, :n_t, g, :]]
            s_parts = [scale * _mm(kp, q[i, h], ordered) for kp in k_parts]
            if sum(len(sp) for sp in s_parts) == 0:
                raise ValueError("no keys to attend to")
            m = max(sp.max() for sp in s_parts if len(sp))
            num, den = np.zeros(d), 0.0
            for sp, vp in zip(s_parts, v_parts):
                w = _exp(sp - m, ordered)
                den += _colsum(w, ordered)
                num += _mm(vp.T, w, ordered)
            out[i, h] = num / den
    return out


def attend_latent(pk, rk, pv, rv, table, q, tail_k, tail_v, tail_len, scale,
                  columns=None, return_weights=False, ordered=False):
    """Same result as attend_dense, computed in each block's rank space.

    For query column (i, h) with KV head g and selected block b:
      (projection)    qt_b = R^K_b[:, g*d:(g+1)*d] q_ih          (length rk_b)
      (scores)        s_bt = scale * P^K_b[t] . qt_b
      (tail scores)   s_tau = scale * tail_k[i, tau, g] . q_ih
      (softmax)       M = max of every score, w = exp(s - M), l = sum of all w
      (latent V)      ot_b = sum_t w_bt P^V_b[t]                (length rv_b)
      (up-projection) u_b = R^V_b[:, g*d:(g+1)*d]^T ot_b
      (tail values)   u_tail = sum_tau w_tau tail_v[i, tau, g]
      (output)        o = (sum_b u_b + u_tail) / l

    columns: optional list of (i, h) pairs to evaluate (default: all).
    Returns o [len(columns), d] when columns is given, else [n_q, H_q, d].
    With return_weights, also returns the normalised weights of every column
    (blocks in table order, tokens ascending, then the tail).  Sums over keys
    run block by block in table order, then over the tail, as in attend_dense;
    ordered=True makes every dot product and sum run left to right.
    """
    n_q, n_q_heads, d, n_kv, G = _shapes(q, [rk[b] for b in table], tail_k)
    all_cols = columns is None
    if all_cols:
        columns = [(i, h) for i in range(n_q) for h in range(n_q_heads)]
    columns = [(int(i), int(h)) for i, h in columns]
    out = np.empty((len(columns), d))
    weights = [None] * len(columns)

    by_group = {}
    for c, (i, h) in enumerate(columns):
        by_group.setdefault(h // G, []).append(c)

    for g, cidx in by_group.items():
        gs = slice(g * d, (g + 1) * d)
        qg = np.stack([q[columns[c][0], columns[c][1]] for c in cidx], axis=1)  # [d, n]
        # scores of every selected block: [T_b, n]
        s_blk = [scale * _mm(pk[b], _mm(rk[b][:, gs], qg, ordered), ordered) for b in table]
        # tail scores per column (each request has its own tail)
        s_tail = []
        for c in cidx:
            i, h = columns[c]
            n_t = int(tail_len[i])
            s_tail.append(scale * _mm(tail_k[i, :n_t, g, :], q[i, h], ordered))
        m = np.full(len(cidx), -np.inf)
        for s in s_blk:
            if s.shape[0]:
                m = np.maximum(m, s.max(axis=0))
        for k, s in enumerate(s_tail):
            if s.shape[0]:
                m[k] = max(m[k], s.max())
        if not np.all(np.isfinite(m)):
            raise ValueError("no keys to attend to")
        w_blk = [_exp(s - m, ordered) for s in s_blk]
        w_tail = [_exp(s - m[k], ordered) for k, s in enumerate(s_tail)]
        l = np.zeros(len(cidx))
        for w in w_blk:
            l += _colsum(w, ordered)
        for k, w in enumerate(w_tail):
            l[k] += _colsum(w, ordered)
        u = np.zeros((d, len(cidx)))
        for b, w in zip(table, w_blk):
            ot = _mm(pv[b].T, w, ordered)              # [rv_b, n]
            u += _mm(rv[b][:, gs].T, ot, ordered)      # [d, n]
        for k, c in enumerate(cidx):
            i, h = columns[c]
            n_t = int(tail_len[i])
            u_tail = _mm(tail_v[i, :n_t, g, :].T, w_tail[k], ordered)
            out[c] = (u[:, k] + u_tail) / l[k]
            if return_weights:
                weights[c] = np.concatenate([w[:, k] for w in w_blk] + [w_tail[k]]) / l[k]

    if all_cols:
        out = out.reshape(n_q, n_q_heads, d)
    return (out, weights) if return_weights else out


def attend_prefill(pk, rk, pv, rv, table, q, tail_k, tail_v, tail_base, scale, key_pos=None, rope_theta=None):
    """Causal prefill of one request (Alg. 1 inference stage with a multi-token
    input query Q, Eq. 1 with the causal mask of an autoregressive model over
    Q's own tokens): token j of the chunk q [n_tok, H_q, d] attends to the
    selected blocks and to the first tail_base + j + 1 rows of the one tail
    tail_k / tail_v [tail_cap, H_kv, d] (the rows before the chunk, then the
    chunk's own tokens up to and including j).  key_pos / rope_theta as for
    attend_dense.  Returns [n_tok, H_q, d]."""
    n_tok = q.shape[0]
    if tail_base + n_tok > tail_k.shape[0]:
        raise ValueError("the tail must hold tail_base + n_tok rows")
    tk = np.broadcast_to(tail_k, (n_tok,) + tail_k.shape)
    tv = np.broadcast_to(tail_v, (n_tok,) + tail_v.shape)
    tail_len = tail_base + 1 + np.arange(n_tok)
    return attend_dense(pk, rk, pv, rv, table, q, tk, tv, tail_len, scale, key_pos=key_pos, rope_theta=rope_theta)


# --------------------------------------------------------------------------
# Rank allocation (Sec. 4.3, Eqs. 5-7)
# --------------------------------------------------------------------------
def spectral_information(sigma, r: int, eps: float) -> float:
    """Eq. 5: H(r) = sum over the r largest singular values of log(1 + sigma^2 / eps^2).
    sigma: one block's singular values, non-increasing."""
    s = np.asarray(sigma, dtype=np.float64)[:r]
    return float(np.sum(np.log1p(s * s / (eps * eps))))


def allocate_ranks(sigmas, r_total: int, r_min: int, r_max: int, eps: float = 1e-3) -> np.ndarray:
    """Eq. 6 solved by the greedy of Eq. 7: every block starts at r_min; each
    remaining rank unit goes to the block whose next singular value brings the
    largest gain log(1 + sigma_{i,r+1}^2 / eps^2); stop when the ranks sum to the
    budget or no block can grow.

    Readings where the text leaves it open: a block cannot take more ranks than
    it has singular values (min(T_b, D)), so its floor is min(r_min, n_i) and its
    cap min(r_max, n_i); if every block reaches its cap first the sum stays below
    the budget (the constraint of Eq. 6 is an inequality); equal gains go to the
    lower block index.

    sigmas: list of 1-D arrays, block i's singular values, non-increasing
    returns int64 ranks [n_blocks]; raises ValueError when even the floors exceed
    the budget (Eq. 6 has no feasible point)."""
    n = len(sigmas)
    sig = [np.asarray(s, dtype=np.float64) for s in sigmas]
    for i, s in enumerate(sig):
        if s.ndim != 1 or np.any(~np.isfinite(s)) or np.any(s < 0) or np.any(np.diff(s) > 0):
            raise ValueError(f"block {i}: singular values must be finite, non-negative, non-increasing")
    cap = np.array([min(r_max, len(s)) for s in sig], dtype=np.int64)
    r = np.array([min(r_min, len(s)) for s in sig], dtype=np.int64)
    if int(r.sum()) > r_total:
        raise ValueError("the budget is below the sum of the per-block floors")

    def gain(i):  # Delta H_{i, r_i}: the gain of block i's next singular value
        if r[i] >= cap[i]:
            return -np.inf
        x = sig[i][r[i]]
        return np.log1p(x * x / (eps * eps))

    nxt = np.array([gain(i) for i in range(n)])
    left = r_total - int(r.sum())
    while left > 0:
        i = int(np.argmax(nxt))          # first index among equal maxima
        if nxt[i] == -np.inf:
            break                        # every block is at its cap
        r[i] += 1
        left -= 1
        nxt[i] = gain(i)
    return r


# --------------------------------------------------------------------------
# INT8 P factors (Sec. 5.3, Table 2: the low-rank cache combined with INT8)
# --------------------------------------------------------------------------
def quantize_rows_int8(p):
    """Symmetric INT8 quantisation of a P factor with one scale per token row:
    s_t = max_k |P[t][k]| / 127 and c[t][k] = P[t][k] / s_t rounded to the
    nearest integer, ties to even, both computed in fp32 (P holds bf16 values,
    exact in fp32; fp32 division is correctly rounded); a row of zeros gets
    s = 0 and codes 0.  Returns (codes int8 [T][r], scales float32 [T]); the
    factor the attention then uses is dequantize_rows_int8(codes, scales)."""
    p = np.asarray(p, dtype=np.float32)
    if p.ndim != 2:
        raise ValueError("P must be 2-D")
    amax = np.abs(p).max(axis=1) if p.shape[1] else np.zeros(p.shape[0], np.float32)
    if not np.all(np.isfinite(amax)):
        raise ValueError("P must be finite")
    scales = (amax / np.float32(127.0)).astype(np.float32)
    codes = np.zeros(p.shape, dtype=np.int8)
    nz = scales > 0
    q = np.rint(p[nz] / scales[nz, None])          # fp32 / fp32 -> fp32, then ties to even
    codes[nz] = np.clip(q, -127, 127).astype(np.int8)
    return codes, scales


def dequantize_rows_int8(codes, scales):
    """The factor INT8 storage stands for: P[t][k] = s_t c[t][k] (float64, exact)."""
    return np.asarray(scales, dtype=np.float64)[:, None] * np.asarray(codes, dtype=np.float64)


# --------------------------------------------------------------------------
# Per-block truncated SVD of the encoder (Sec. 4.2 Eq. 3, Alg. 1 encoding stage)
# --------------------------------------------------------------------------
def block_svd(k, tol: float = 1e-13, max_sweeps: int = 60):
    """Singular values and right singular vectors of one block's K (T x D), by
    one-sided Jacobi (Hestenes): rotate pairs of columns of A = K until every
    pair is orthogonal; the rotations accumulate into V, the column norms of
    the final A are the singular values.  Textbook cyclic order (p < q, row by
    row), fp64.  Returns (sigma [D] non-increasing, V [D, D] with column j the
    right singular vector of sigma_j), so K = U diag(sigma) V^T with
    U = A / sigma.  Only the first min(T, D) values can be non-zero."""
    a = np.array(k, dtype=np.float64)
    n = a.shape[1]
    v = np.eye(n)
    for _ in range(max_sweeps):
        rotated = False
        for p in range(n - 1):
            for q in range(p + 1, n):
                alpha = a[:, p] @ a[:, p]
                beta = a[:, q] @ a[:, q]
                gamma = a[:, p] @ a[:, q]
                if gamma == 0.0 or abs(gamma) <= tol * math.sqrt(alpha * beta):
                    continue
                rotated = True
                # the rotation that makes columns p and q orthogonal
                zeta = (beta - alpha) / (2.0 * gamma)
                t = math.copysign(1.0, zeta) / (abs(zeta) + math.sqrt(1.0 + zeta * zeta))
                c = 1.0 / math.sqrt(1.0 + t * t)
                s_ = c * t
                ap, aq = a[:, p].copy(), a[:, q].copy()
                a[:, p], a[:, q] = c * ap - s_ * aq, s_ * ap + c * aq
                vp, vq = v[:, p].copy(), v[:, q].copy()
                v[:, p], v[:, q] = c * vp - s_ * vq, s_ * vp + c * vq
        if not rotated:
            break
    sigma = np.sqrt(np.sum(a * a, axis=0))
    order = np.argsort(-sigma, kind="stable")
    return sigma[order], v[:, order]


def block_factors(k, v, r: int):
    """Eq. 3 truncated at rank r with the singular values folded into P:
    P = U_r Sigma_r = K V_r (T x r) and R = V_r^T (r x D), so P R is the best
    rank-r approximation of K."""
    vr = np.asarray(v, dtype=np.float64)[:, :r]
    return np.asarray(k, dtype=np.float64) @ vr, vr.T.copy()
