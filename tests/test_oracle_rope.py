"""Pins of the oracle's rotary position embedding and of its pre-RoPE attention
(CPU).  The rotation is checked against the Qwen2 implementation in the installed
transformers package (its frequencies and its rotate-half routine), against a
complex-number formulation written here, and by the properties that any rotary
embedding has: it preserves pair norms, is the identity at position 0, composes
additively, and makes scores depend on the position difference only."""
import numpy as np
import pytest

import oracle

THETA = 1e6  # Qwen2.5's base


def _complex_rope(x, pos, theta):
    """The same rotation written as complex multiplication: pair j of a row is
    the complex number x_j + i x_{j+d/2}, multiplied by exp(i p omega_j),
    omega_j = exp(-(2j/d) ln theta)."""
    d = x.shape[-1]
    z = x[..., : d // 2] + 1j * x[..., d // 2:]
    omega = np.exp(-(2.0 * np.arange(d // 2) / d) * np.log(theta))
    rot = np.exp(1j * np.multiply.outer(np.asarray(pos, dtype=np.float64), omega))
    rot = rot.reshape(rot.shape[:1] + (1,) * (x.ndim - 2) + rot.shape[1:])
    w = z * rot
    return np.concatenate([w.real, w.imag], axis=-1)


@pytest.mark.parametrize("d", [64, 128])
def test_rope_matches_the_qwen2_implementation(d):
    torch = pytest.importorskip("torch")
    tr = pytest.importorskip("transformers")
    from transformers.models.qwen2 import modeling_qwen2 as qm
    cfg = tr.Qwen2Config(hidden_size=8 * d, num_attention_heads=8, num_key_value_heads=2, head_dim=d,
                         rope_parameters={"rope_type": "default", "rope_theta": THETA},
                         max_position_embeddings=4096)
    emb = qm.Qwen2RotaryEmbedding(cfg)
    rng = np.random.default_rng(d)
    T, H = 64, 3
    pos = np.sort(rng.choice(2048, T, replace=False))
    x = rng.standard_normal((T, H, d))
    cos, sin = emb(torch.zeros(1, T, d), torch.from_numpy(pos)[None])      # fp32 [1, T, d]
    xt = torch.from_numpy(x.transpose(1, 0, 2)[None])                      # [1, H, T, d]
    qr, _ = qm.apply_rotary_pos_emb(xt, xt, cos.double(), sin.double())
    ref = qr[0].numpy().transpose(1, 0, 2)
    got = oracle.rope(x, pos, THETA)
    # the library forms its angles in fp32 (positions below 2048: < 3e-4 rad)
    assert np.abs(got - ref).max() < 2e-3
    # a dropped sign, swapped pairing or a wrong frequency exponent is O(1)
    assert np.abs(oracle.rope(x, pos, THETA * 10) - ref).max() > 0.1


def test_rope_matches_complex_multiplication():
    rng = np.random.default_rng(1)
    x = rng.standard_normal((40, 2, 128))
    pos = rng.integers(0, 1 << 21, 40)
    np.testing.assert_allclose(oracle.rope(x, pos, THETA), _complex_rope(x, pos, THETA), rtol=0, atol=1e-9)


def test_rope_properties():
    rng = np.random.default_rng(2)
    d = 64
    x = rng.standard_normal((30, d))
    a = rng.integers(0, 1 << 20, 30)
    b = rng.integers(0, 1 << 20, 30)
    y = oracle.rope(x, a, THETA)
    # each pair keeps its norm
    np.testing.assert_allclose(np.hypot(y[:, : d // 2], y[:, d // 2:]), np.hypot(x[:, : d // 2], x[:, d // 2:]),
                               rtol=1e-12)
    # position 0 is the identity, bit for bit (cos 0 = 1, sin 0 = 0)
    assert np.array_equal(oracle.rope(x, np.zeros(30, np.int64), THETA), x)
    # rotations compose additively
    np.testing.assert_allclose(oracle.rope(y, b, THETA), oracle.rope(x, a + b, THETA), rtol=0, atol=1e-8)
    # scores depend on the position difference only
    q = rng.standard_normal((30, d))
    lhs = np.einsum("td,td->t", oracle.rope(q, a, THETA), oracle.rope(x, b, THETA))
    rhs = np.einsum("td,td->t", oracle.rope(q, a - b, THETA), x)
    np.testing.assert_allclose(lhs, rhs, rtol=0, atol=1e-8)


def _case(seed, d=64, n_kv=2, G=2, n_q=2, T=(40, 25), r=(6, 9), tail=5):
    rng = np.random.default_rng(seed)
    D = n_kv * d
    pk = [rng.standard_normal((t, k)) for t, k in zip(T, r)]
    rk = [rng.standard_normal((k, D)) / np.sqrt(k) for k in r]
    pv = [rng.standard_normal((t, k)) for t, k in zip(T, r)]
    rv = [rng.standard_normal((k, D)) / np.sqrt(k) for k in r]
    q = rng.standard_normal((n_q, n_kv * G, d))
    tk = rng.standard_normal((n_q, tail, n_kv, d))
    tv = rng.standard_normal((n_q, tail, n_kv, d))
    return pk, rk, pv, rv, q, tk, tv, np.array([tail, tail - 2]), 1 / np.sqrt(d)


def test_rope_attention_at_position_zero_is_plain_attention():
    pk, rk, pv, rv, q, tk, tv, tl, sc = _case(3)
    table = [1, 0]
    plain = oracle.attend_dense(pk, rk, pv, rv, table, q, tk, tv, tl, sc)
    # a one-token block at position 0 keeps its key exactly
    pk0 = [p[:1] for p in pk]
    pv0 = [p[:1] for p in pv]
    got = oracle.attend_dense(pk0, rk, pv0, rv, table, q, tk, tv, tl, sc, key_pos=[0, 0], rope_theta=THETA)
    ref = oracle.attend_dense(pk0, rk, pv0, rv, table, q, tk, tv, tl, sc)
    assert np.array_equal(got, ref)
    # longer blocks move: the rotation is really applied
    moved = oracle.attend_dense(pk, rk, pv, rv, table, q, tk, tv, tl, sc, key_pos=[0, 0], rope_theta=THETA)
    assert np.abs(moved - plain).max() > 1e-3


def test_rope_attention_equals_attention_over_rotated_keys():
    """Block b's token t sits at key_pos[b] + t: the same attention as over
    uncompressed blocks whose keys were rotated by the complex formulation."""
    d, n_kv = 64, 2
    pk, rk, pv, rv, q, tk, tv, tl, sc = _case(4, d=d, n_kv=n_kv)
    key_pos = [1000, 77]
    table = [0, 1]
    got = oracle.attend_dense(pk, rk, pv, rv, table, q, tk, tv, tl, sc, key_pos=key_pos, rope_theta=THETA)
    D = n_kv * d
    k_rot = []
    for b in range(2):
        k = (pk[b] @ rk[b]).reshape(-1, n_kv, d)
        k_rot.append(_complex_rope(k, key_pos[b] + np.arange(k.shape[0]), THETA).reshape(-1, D))
    eye = [np.eye(D)] * 2
    ref = oracle.attend_dense(k_rot, eye, pv, rv, table, q, tk, tv, tl, sc)
    np.testing.assert_allclose(got, ref, rtol=0, atol=1e-10)


def test_rope_attention_is_shift_invariant():
    """Moving every key and the query by the same number of positions changes
    no score: blocks shifted by delta, the (already rotated) query and tail keys
    rotated by delta more, give the same output."""
    pk, rk, pv, rv, q, tk, tv, tl, sc = _case(5)
    delta = 123457
    key_pos = [300, 5]
    a = oracle.attend_dense(pk, rk, pv, rv, [0, 1], q, tk, tv, tl, sc, key_pos=key_pos, rope_theta=THETA)
    rot = lambda x: oracle.rope(x.reshape(-1, x.shape[-1]), np.full(x.size // x.shape[-1], delta), THETA).reshape(
        x.shape)
    b = oracle.attend_dense(pk, rk, pv, rv, [0, 1], rot(q), rot(tk), tv, tl, sc,
                            key_pos=[p + delta for p in key_pos], rope_theta=THETA)
    np.testing.assert_allclose(a, b, rtol=0, atol=1e-9)
    # a shift of the blocks alone is not invisible
    c = oracle.attend_dense(pk, rk, pv, rv, [0, 1], q, tk, tv, tl, sc, key_pos=[p + delta for p in key_pos],
                            rope_theta=THETA)
    assert np.abs(a - c).max() > 1e-3
