"""Pins for the CPU oracle.

Every pin checks the oracle against something other than itself: a library
routine (torch's scaled_dot_product_attention) on a special case that reduces
to plain attention, pure-Python brute force on tiny inputs, closed forms,
invariances of the mathematics, and a hand-derived worked example.  The last
test plants plausible mistakes in a copy of the oracle (on the CPU) and checks
that each one fails at least one pin that does not merely compare the oracle's
two routes with each other.
"""
import inspect
import math
import os

import numpy as np
import pytest
import torch

import oracle
from helpers import oracle_args
from synth import make_problem

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "rank1_blocks_with_tail.txt")


def _col_rel(a, b):
    a = np.asarray(a).reshape(-1, np.shape(b)[-1])
    b = np.asarray(b).reshape(-1, np.shape(b)[-1])
    return float(np.max(np.linalg.norm(a - b, axis=1) / np.maximum(np.linalg.norm(b, axis=1), 1e-300)))


def _case(seed, block_tokens, rank_k, rank_v=None, **kw):
    return oracle_args(make_problem(seed, block_tokens, rank_k, rank_v, **kw))


CASES = [
    dict(block_tokens=[1, 3, 17], rank_k=[1, 2, 5], rank_v=[1, 4, 3], n_kv_heads=2, head_dim=4,
         n_q=2, n_q_heads=4, tail_cap=5, tail_len=[5, 2]),
    dict(block_tokens=[7], rank_k=[8], rank_v=[8], n_kv_heads=1, head_dim=8, n_q=1, n_q_heads=3,
         tail_cap=0),
    dict(block_tokens=[4, 9], rank_k=[6, 6], rank_v=[2, 6], n_kv_heads=3, head_dim=2, n_q=3,
         n_q_heads=6, tail_cap=4, tail_len=[0, 4, 1]),
]


def _sdpa(q_vec, keys, vals, scale):
    """torch's attention on one query row (fp64, CPU)."""
    qt = torch.from_numpy(np.asarray(q_vec, dtype=np.float64)).view(1, 1, 1, -1)
    kt = torch.from_numpy(np.asarray(keys, dtype=np.float64)).view(1, 1, keys.shape[0], -1)
    vt = torch.from_numpy(np.asarray(vals, dtype=np.float64)).view(1, 1, vals.shape[0], -1)
    return torch.nn.functional.scaled_dot_product_attention(qt, kt, vt, scale=scale).view(-1).numpy()


# ----------------------------------------------------------------------------------
# pins: each takes (dense, latent) implementations and raises AssertionError on failure
# ----------------------------------------------------------------------------------
def pin_cross_routes(dense, latent):
    """Not external: the two routes must agree (exact reassociation)."""
    for k, c in enumerate(CASES):
        a = _case(10 + k, **c)
        assert _col_rel(latent(**a), dense(**a)) < 1e-12


def pin_identity_factors_sdpa(dense, latent):
    """P = K, R = I at full rank (r = H_kv*d): the method reduces to plain attention."""
    rng = np.random.default_rng(1)
    n_kv, d, n_q, n_q_heads = 2, 4, 2, 4
    D, G = n_kv * d, n_q_heads // n_kv
    T = [3, 5]
    K = [rng.standard_normal((t, D)) for t in T]
    V = [rng.standard_normal((t, D)) for t in T]
    eye = np.eye(D)
    q = rng.standard_normal((n_q, n_q_heads, d))
    tk = rng.standard_normal((n_q, 2, n_kv, d))
    tv = rng.standard_normal((n_q, 2, n_kv, d))
    tl = np.array([2, 1])
    args = dict(pk=K, rk=[eye, eye], pv=V, rv=[eye, eye], table=[0, 1], q=q, tail_k=tk,
                tail_v=tv, tail_len=tl, scale=0.7)
    od, ol = dense(**args), latent(**args)
    for i in range(n_q):
        for h in range(n_q_heads):
            g = h // G
            keys = np.concatenate([K[0][:, g * d:(g + 1) * d], K[1][:, g * d:(g + 1) * d], tk[i, :tl[i], g]])
            vals = np.concatenate([V[0][:, g * d:(g + 1) * d], V[1][:, g * d:(g + 1) * d], tv[i, :tl[i], g]])
            ref = _sdpa(q[i, h], keys, vals, 0.7)
            assert np.allclose(od[i, h], ref, rtol=1e-12, atol=1e-13)
            assert np.allclose(ol[i, h], ref, rtol=1e-12, atol=1e-13)


def test_identity_factors_routes_agree_bitwise():
    """P = K, R = I at full rank (r = H_kv*d), with every sum taken left to right
    (ordered=True): the latent route's projection multiplies by 1 and adds exact
    zeros, its up-projection selects the head's rows of the latent sums, and both
    routes group the softmax sums block by block in table order, then the tail.
    So the two routes are not merely close: they agree to the last bit, and the
    latent route equals plain attention over K and V exactly."""
    rng = np.random.default_rng(31)
    for n_kv, d, G, T, tl in ((2, 4, 2, [3, 5], [2, 1]), (1, 8, 3, [7], [0, 4]), (3, 2, 1, [1, 6, 2], [3, 3])):
        D, n_q = n_kv * d, len(tl)
        K = [rng.standard_normal((t, D)) for t in T]
        V = [rng.standard_normal((t, D)) for t in T]
        eye = np.eye(D)
        args = dict(pk=K, rk=[eye] * len(T), pv=V, rv=[eye] * len(T), table=list(range(len(T)))[::-1],
                    q=rng.standard_normal((n_q, n_kv * G, d)), tail_k=rng.standard_normal((n_q, 4, n_kv, d)),
                    tail_v=rng.standard_normal((n_q, 4, n_kv, d)), tail_len=np.array(tl), scale=0.45)
        od = oracle.attend_dense(**args, ordered=True)
        ol = oracle.attend_latent(**args, ordered=True)
        assert np.array_equal(od.view(np.uint64), ol.view(np.uint64))
        # and the BLAS route agrees with the ordered one within rounding
        assert _col_rel(oracle.attend_latent(**args), ol) < 1e-13


def pin_bruteforce_tiny(dense, latent):
    """Scalar Python loops: rebuild every key/value element, softmax with math.exp."""
    a = _case(3, [2, 3], [2, 1], [1, 2], n_kv_heads=2, head_dim=2, n_q=2, n_q_heads=4,
              tail_cap=2, tail_len=[1, 2])
    pk, rk, pv, rv, q = a["pk"], a["rk"], a["pv"], a["rv"], a["q"]
    tk, tv, tl, sc = a["tail_k"], a["tail_v"], a["tail_len"], a["scale"]
    n_q, n_q_heads, d = q.shape
    G = n_q_heads // 2
    ref = np.zeros_like(q)
    for i in range(n_q):
        for h in range(n_q_heads):
            g = h // G
            keys, vals = [], []
            for b in a["table"]:
                for t in range(pk[b].shape[0]):
                    keys.append([sum(pk[b][t][k] * rk[b][k][g * d + j] for k in range(pk[b].shape[1]))
                                 for j in range(d)])
                    vals.append([sum(pv[b][t][k] * rv[b][k][g * d + j] for k in range(pv[b].shape[1]))
                                 for j in range(d)])
            for t in range(int(tl[i])):
                keys.append(list(tk[i, t, g]))
                vals.append(list(tv[i, t, g]))
            s = [sc * sum(kk[j] * q[i, h, j] for j in range(d)) for kk in keys]
            mx = max(s)
            e = [math.exp(x - mx) for x in s]
            tot = sum(e)
            for j in range(d):
                ref[i, h, j] = sum(e[t] * vals[t][j] for t in range(len(e))) / tot
    assert _col_rel(dense(**a), ref) < 1e-12
    assert _col_rel(latent(**a), ref) < 1e-12


def pin_q_zero_closed_form(dense, latent):
    """q = 0: every key gets weight 1/n, so o is the mean value row, computed here
    from column sums of P^V: (sum_b (1^T P^V_b) R^V_b[:, g] + sum_t tail_v) / n."""
    c = CASES[0]
    a = _case(4, **c)
    a["q"] = np.zeros_like(a["q"])
    n_q, n_q_heads, d = a["q"].shape
    G = n_q_heads // a["tail_k"].shape[2]
    n_ctx = sum(a["pk"][b].shape[0] for b in a["table"])
    for impl in (dense, latent):
        o = impl(**a)
        for i in range(n_q):
            for h in range(n_q_heads):
                g = h // G
                acc = sum(a["pv"][b].sum(axis=0) @ a["rv"][b][:, g * d:(g + 1) * d] for b in a["table"])
                acc = acc + a["tail_v"][i, :a["tail_len"][i], g].sum(axis=0)
                assert np.allclose(o[i, h], acc / (n_ctx + a["tail_len"][i]), rtol=1e-12, atol=1e-14)


def pin_weights(dense, latent):
    """Softmax weights sum to 1; at q = 0 they are exactly uniform."""
    a = _case(5, **CASES[2])
    _, w = latent(**a, return_weights=True)
    for wc in w:
        assert abs(wc.sum() - 1.0) < 1e-14 * len(wc)
    a["q"] = np.zeros_like(a["q"])
    _, w = latent(**a, return_weights=True)
    for wc in w:
        assert np.all(wc == wc[0])


def pin_orthogonal_invariance(dense, latent):
    """P -> P M, R -> M^T R with M orthogonal leaves K, V and the output unchanged."""
    a = _case(6, **CASES[0])
    o0 = (dense(**a), latent(**a))
    rng = np.random.default_rng(7)
    b = dict(a)
    for key_p, key_r in (("pk", "rk"), ("pv", "rv")):
        ps, rs = [], []
        for p, r in zip(a[key_p], a[key_r]):
            m, _ = np.linalg.qr(rng.standard_normal((p.shape[1], p.shape[1])))
            ps.append(p @ m)
            rs.append(m.T @ r)
        b[key_p], b[key_r] = ps, rs
    assert _col_rel(dense(**b), o0[0]) < 1e-12
    assert _col_rel(latent(**b), o0[1]) < 1e-12


def pin_permutation_and_split(dense, latent):
    """Block order does not matter; splitting a block's rows into two blocks with
    the same R gives the same output."""
    a = _case(8, **CASES[0])
    ref = dense(**a)
    perm = dict(a, table=a["table"][::-1])
    assert _col_rel(dense(**perm), ref) < 1e-12
    assert _col_rel(latent(**perm), ref) < 1e-12
    b = dict(a)
    cut = 9
    b["pk"] = a["pk"][:2] + [a["pk"][2][:cut], a["pk"][2][cut:]]
    b["pv"] = a["pv"][:2] + [a["pv"][2][:cut], a["pv"][2][cut:]]
    b["rk"] = a["rk"][:2] + [a["rk"][2], a["rk"][2]]
    b["rv"] = a["rv"][:2] + [a["rv"][2], a["rv"][2]]
    b["table"] = [0, 1, 2, 3]
    assert _col_rel(dense(**b), ref) < 1e-12
    assert _col_rel(latent(**b), ref) < 1e-12


def pin_tail_only_sdpa(dense, latent):
    """No selected blocks: plain attention of each request over its own tail."""
    a = _case(9, [4], [2], n_kv_heads=2, head_dim=8, n_q=3, n_q_heads=4, tail_cap=6,
              tail_len=[6, 1, 3])
    a["table"] = []
    for impl in (dense, latent):
        o = impl(**a)
        for i in range(3):
            for h in range(4):
                g = h // 2
                n = a["tail_len"][i]
                ref = _sdpa(a["q"][i, h], a["tail_k"][i, :n, g], a["tail_v"][i, :n, g], a["scale"])
                assert np.allclose(o[i, h], ref, rtol=1e-12, atol=1e-14)


def pin_single_key_and_gqa(dense, latent):
    """One key in total: every head returns that key's value row, and head h reads
    KV head floor(h / G) (the value's head slices are distinct)."""
    d, n_kv, n_q_heads = 3, 3, 6
    D = n_kv * d
    rng = np.random.default_rng(11)
    pk, rk = [rng.standard_normal((1, 2))], [rng.standard_normal((2, D))]
    pv, rv = [rng.standard_normal((1, 2))], [rng.standard_normal((2, D))]
    q = rng.standard_normal((1, n_q_heads, d))
    tk = np.zeros((1, 0, n_kv, d))
    args = dict(pk=pk, rk=rk, pv=pv, rv=rv, table=[0], q=q, tail_k=tk, tail_v=tk,
                tail_len=np.array([0]), scale=0.3)
    v_row = pv[0][0] @ rv[0]
    for impl in (dense, latent):
        o = impl(**args)
        for h in range(n_q_heads):
            g = h // 2
            assert np.allclose(o[0, h], v_row[g * d:(g + 1) * d], rtol=1e-13, atol=1e-15)
    # the same through the tail alone, one token
    tk1 = rng.standard_normal((1, 1, n_kv, d))
    tv1 = rng.standard_normal((1, 1, n_kv, d))
    args2 = dict(args, table=[], tail_k=tk1, tail_v=tv1, tail_len=np.array([1]))
    for impl in (dense, latent):
        o = impl(**args2)
        for h in range(n_q_heads):
            assert np.allclose(o[0, h], tv1[0, 0, h // 2], rtol=1e-13, atol=1e-15)


def pin_two_key_closed_form(dense, latent):
    """Two keys: weights are logistic in the score gap scale*(q.k1 - q.k2)."""
    d = 4
    rng = np.random.default_rng(12)
    k1, k2 = rng.standard_normal(d), rng.standard_normal(d)
    v1, v2 = rng.standard_normal(d), rng.standard_normal(d)
    qv = rng.standard_normal(d)
    sc = 0.37
    # block 0 holds key/value 1 as a rank-1 factorisation; key/value 2 is the tail
    args = dict(pk=[np.array([[2.0]])], rk=[k1[None, :] / 2.0], pv=[np.array([[0.5]])],
                rv=[v1[None, :] * 2.0], table=[0], q=qv.reshape(1, 1, d),
                tail_k=k2.reshape(1, 1, 1, d), tail_v=v2.reshape(1, 1, 1, d),
                tail_len=np.array([1]), scale=sc)
    gap = sc * (qv @ k1 - qv @ k2)
    w1 = 1.0 / (1.0 + math.exp(-gap))
    ref = w1 * v1 + (1.0 - w1) * v2
    for impl in (dense, latent):
        assert np.allclose(impl(**args)[0, 0], ref, rtol=1e-13, atol=1e-15)


def _load_golden():
    blocks, fields = [], {}
    with open(GOLDEN) as f:
        for line in f:
            line = line.split("#", 1)[0].split()
            if not line:
                continue
            key, vals = line[0], [float(x) for x in line[1:]]
            if key == "block":
                blocks.append({"tokens": int(vals[0]), "rank_k": int(vals[1]), "rank_v": int(vals[2])})
            elif key in ("pk", "rk", "pv", "rv"):
                blocks[-1][key] = vals
            else:
                fields[key] = vals
    return blocks, fields


def pin_golden(dense, latent):
    blocks, f = _load_golden()
    n_q_heads, n_kv, d = int(f["n_q_heads"][0]), int(f["n_kv_heads"][0]), int(f["head_dim"][0])
    D = n_kv * d
    pk = [np.array(b["pk"]).reshape(b["tokens"], b["rank_k"]) for b in blocks]
    rk = [np.array(b["rk"]).reshape(b["rank_k"], D) for b in blocks]
    pv = [np.array(b["pv"]).reshape(b["tokens"], b["rank_v"]) for b in blocks]
    rv = [np.array(b["rv"]).reshape(b["rank_v"], D) for b in blocks]
    n_t = len(f["tail_k"]) // D
    args = dict(pk=pk, rk=rk, pv=pv, rv=rv, table=list(range(len(blocks))),
                q=np.array(f["q"]).reshape(1, n_q_heads, d),
                tail_k=np.array(f["tail_k"]).reshape(1, n_t, n_kv, d),
                tail_v=np.array(f["tail_v"]).reshape(1, n_t, n_kv, d),
                tail_len=np.array([n_t]), scale=f["scale"][0])
    expect = np.array(f["expect"]).reshape(1, n_q_heads, d)
    for impl in (dense, latent):
        for table in ([0, 1], [1, 0]):
            assert np.allclose(impl(**dict(args, table=table)), expect, rtol=1e-14, atol=1e-14)


EXTERNAL_PINS = [pin_identity_factors_sdpa, pin_bruteforce_tiny, pin_q_zero_closed_form,
                 pin_weights, pin_orthogonal_invariance, pin_permutation_and_split,
                 pin_tail_only_sdpa, pin_single_key_and_gqa, pin_two_key_closed_form, pin_golden]


@pytest.mark.parametrize("pin", [pin_cross_routes] + EXTERNAL_PINS, ids=lambda p: p.__name__)
def test_pin(pin):
    pin(oracle.attend_dense, oracle.attend_latent)


def test_columns_subset_matches_full():
    a = _case(13, **CASES[2])
    full = oracle.attend_latent(**a)
    cols = [(2, 5), (0, 0), (1, 3)]
    sub = oracle.attend_latent(**a, columns=cols)
    for k, (i, h) in enumerate(cols):
        assert np.allclose(sub[k], full[i, h], rtol=1e-14, atol=1e-15)


def test_no_keys_is_an_error():
    a = _case(14, [3], [2], n_kv_heads=1, head_dim=2, n_q=1, n_q_heads=1, tail_cap=2, tail_len=[0])
    a["table"] = []
    with pytest.raises(ValueError):
        oracle.attend_dense(**a)
    with pytest.raises(ValueError):
        oracle.attend_latent(**a)


# ----------------------------------------------------------------------------------
# planted mistakes (in a copy of the oracle, on the CPU) must fail an external pin
# ----------------------------------------------------------------------------------
MUTATIONS = [
    ("latent: wrong GQA group", "by_group.setdefault(h // G", "by_group.setdefault(h % G"),
    ("dense: wrong GQA group", "g = h // G\n            cols = slice", "g = h % G\n            cols = slice"),
    ("latent: wrong head slice", "gs = slice(g * d, (g + 1) * d)", "gs = slice(g, g + d)"),
    ("dense: wrong head slice", "k_parts = [k[:, cols] for k in keys]", "k_parts = [k[:, g:g + d] for k in keys]"),
    ("latent: scale dropped", "s_blk = [scale * _mm(pk[b]", "s_blk = [_mm(pk[b]"),
    ("dense: scale dropped", "s_parts = [scale * _mm(kp,", "s_parts = [_mm(kp,"),
    ("latent: tail values dropped", "out[c] = (u[:, k] + u_tail) / l[k]", "out[c] = u[:, k] / l[k]"),
    ("latent: tail missing from normaliser", "l[k] += _colsum(w, ordered)", "l[k] += 0.0"),
    ("latent: scores from P^V", "scale * _mm(pk[b],", "scale * _mm(pv[b],"),
    ("latent: latent V from P^K", "ot = _mm(pv[b].T, w, ordered)", "ot = _mm(pk[b].T, w, ordered)"),
    ("latent: up-projection through R^K", "u += _mm(rv[b][:, gs].T, ot, ordered)", "u += _mm(rk[b][:, gs].T, ot, ordered)"),
    ("dense: tail of the wrong request", "+ [tail_k[i, :n_t, g, :]]", "+ [tail_k[0, :n_t, g, :]]"),
    ("dense: values rebuilt with R^K", "vals = [reconstruct(pv[b], rv[b]", "vals = [reconstruct(pv[b], rk[b]"),
    ("latent: tail scores unscaled", "s_tail.append(scale * _mm(", "s_tail.append(1.0 * _mm("),
    ("reconstruct: dropped factor", "return _mm(p, r, ordered)", "return _mm(p, 0.5 * r, ordered)"),
]


@pytest.mark.parametrize("name,old,new", MUTATIONS, ids=[m[0] for m in MUTATIONS])
def test_planted_mistake_is_caught(name, old, new):
    src = inspect.getsource(oracle)
    assert src.count(old) == 1, f"mutation anchor not unique: {old!r}"
    ns = {"__name__": "oracle_mutant"}
    exec(compile(src.replace(old, new), "oracle_mutant", "exec"), ns)
    failed = []
    for pin in EXTERNAL_PINS:
        try:
            pin(ns["attend_dense"], ns["attend_latent"])
        except Exception:  # an assertion or a crash both expose the mistake
            failed.append(pin.__name__)
    assert failed, f"planted mistake '{name}' passed every external pin"


# ----------------------------------------------------------------------------------
# prefill (a multi-token query of one request, causal over its own tokens)
# ----------------------------------------------------------------------------------
def _prefill_case(seed, n_tok, tail_base, extra_rows, n_kv=2, G=3, d=16, blocks=((4, 2), (9, 5))):
    """A prefill problem: blocks (T_b, r_b), one shared tail of tail_base + n_tok
    + extra_rows rows, n_tok query tokens."""
    tail_cap = tail_base + n_tok + extra_rows
    base = _case(seed, [t for t, _ in blocks] or [1], [r for _, r in blocks] or [1],
                 n_kv_heads=n_kv, head_dim=d, n_q=n_tok, n_q_heads=n_kv * G, tail_cap=tail_cap)
    args = {k: base[k] for k in ("pk", "rk", "pv", "rv", "q", "scale")}
    args["table"] = list(range(len(blocks)))
    args["tail_k"], args["tail_v"] = base["tail_k"][0], base["tail_v"][0]  # request 0's tail, shared
    args["tail_base"] = tail_base
    return args


def _causal_sdpa(a, n_tok, G):
    """torch's attention of the chunk over the shared tail with the causal mask
    (fp64, CPU; KV heads repeated for the GQA groups)."""
    tail_base = a["tail_base"]
    n_keys = tail_base + n_tok
    q = torch.from_numpy(np.ascontiguousarray(a["q"].transpose(1, 0, 2)))[None]       # [1, H_q, n_tok, d]
    k = torch.from_numpy(np.ascontiguousarray(a["tail_k"][:n_keys].transpose(1, 0, 2)))
    v = torch.from_numpy(np.ascontiguousarray(a["tail_v"][:n_keys].transpose(1, 0, 2)))
    k = k.repeat_interleave(G, dim=0)[None]
    v = v.repeat_interleave(G, dim=0)[None]
    if tail_base == 0:
        o = torch.nn.functional.scaled_dot_product_attention(q, k, v, scale=a["scale"], is_causal=True)
    else:
        mask = torch.arange(n_keys)[None, :] < (tail_base + 1 + torch.arange(n_tok))[:, None]
        o = torch.nn.functional.scaled_dot_product_attention(q, k, v, attn_mask=mask, scale=a["scale"])
    return o[0].numpy().transpose(1, 0, 2)


@pytest.mark.parametrize("tail_base,extra", [(0, 0), (5, 3)])
def test_prefill_tail_only_matches_causal_sdpa(tail_base, extra):
    """No blocks: the chunk's attention over its tail is textbook causal attention
    (torch's is_causal when the chunk is the whole tail; an explicit mask with
    earlier rows); rows past tail_base + n_tok are never read."""
    n_tok, G = 7, 3
    a = _prefill_case(21, n_tok, tail_base, extra, G=G)
    a["table"] = []
    ref = _causal_sdpa(a, n_tok, G)
    o = oracle.attend_prefill(**a)
    assert np.allclose(o, ref, rtol=1e-12, atol=1e-14)
    a["tail_k"] = a["tail_k"].copy()
    a["tail_k"][tail_base + n_tok:] = 1e6  # unused rows
    assert np.array_equal(oracle.attend_prefill(**a), o)


def test_prefill_token_rows_match_latent_route():
    """With blocks: token j of the chunk is a decode query whose tail is the
    shared tail's first tail_base + j + 1 rows (checked through the latent route,
    which shares no code with the dense definition the prefill wrapper uses)."""
    n_tok, tail_base = 5, 4
    a = _prefill_case(22, n_tok, tail_base, 2)
    o = oracle.attend_prefill(**a)
    for j in range(n_tok):
        ref = oracle.attend_latent(a["pk"], a["rk"], a["pv"], a["rv"], a["table"], a["q"][j:j + 1],
                                   a["tail_k"][None], a["tail_v"][None], [tail_base + j + 1], a["scale"])
        assert _col_rel(o[j:j + 1], ref) < 1e-12
