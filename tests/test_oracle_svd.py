"""Pins for the oracle's per-block truncated SVD (Sec. 4.2 Eq. 3): singular
values against LAPACK (numpy.linalg.svd) on random, wide, tall and
rank-deficient blocks; orthonormal V; K = U diag(sigma) V^T; the Eckart-Young
closed form for the truncation error of P R; a diagonal block and a rank-one
block whose SVDs are known by hand.  Planted mistakes in a copy of the oracle
each fail a pin."""
import inspect
import math

import numpy as np
import pytest

import oracle


def _blocks():
    rng = np.random.default_rng(5)
    yield rng.standard_normal((40, 12))                      # tall
    yield rng.standard_normal((7, 16))                       # wide: only 7 non-zero values
    u, _ = np.linalg.qr(rng.standard_normal((30, 10)))
    w, _ = np.linalg.qr(rng.standard_normal((10, 10)))
    yield u @ np.diag(2.0 ** -np.arange(10)) @ w.T           # spread spectrum
    z = rng.standard_normal((20, 9))
    z[:, 4] = 0.0
    z[:, 7] = 2.0 * z[:, 1]                                  # rank-deficient
    yield z


def pin_lapack_values(svd):
    for k in _blocks():
        sig, _ = svd(k)
        ref = np.linalg.svd(k, compute_uv=False)
        n = min(k.shape)
        assert np.allclose(sig[:n], ref, rtol=1e-10, atol=1e-12 * ref[0])
        assert np.all(sig[n:] <= 1e-10 * ref[0])
        assert np.all(np.diff(sig) <= 0)


def pin_orthonormal_and_reconstruction(svd):
    for k in _blocks():
        sig, v = svd(k)
        assert np.allclose(v.T @ v, np.eye(v.shape[0]), atol=1e-12)
        kv = k @ v                                    # = U diag(sigma): columns of norm sigma
        assert np.allclose(np.linalg.norm(kv, axis=0), sig, rtol=1e-10, atol=1e-12 * sig[0])
        assert np.allclose(kv @ v.T, k, atol=1e-12 * max(1.0, sig[0]))


def pin_eckart_young(svd):
    """||K - P R||_F^2 = sum of the squared singular values past r."""
    for k in _blocks():
        sig, v = svd(k)
        for r in (1, 3, min(k.shape)):
            p, rr = oracle.block_factors(k, v, r)
            err2 = np.sum((k - p @ rr) ** 2)
            assert math.isclose(err2, np.sum(sig[r:] ** 2), rel_tol=1e-9, abs_tol=1e-18 + 1e-12 * sig[0] ** 2)


def pin_hand_examples(svd):
    d = np.zeros((5, 4))
    d[0, 2], d[1, 0], d[3, 3] = -3.0, 5.0, 0.5                # singular values |diag| sorted: 5, 3, 0.5, 0
    sig, v = svd(d)
    assert np.allclose(sig, [5.0, 3.0, 0.5, 0.0], atol=1e-14)
    assert np.allclose(np.abs(v[:, 0]), [1, 0, 0, 0]) and np.allclose(np.abs(v[:, 1]), [0, 0, 1, 0])
    x, y = np.array([1.0, 2.0, 2.0]), np.array([3.0, 0.0, 4.0, 0.0])  # rank one: sigma = |x| |y| = 15
    sig, v = svd(np.outer(x, y))
    assert math.isclose(sig[0], 15.0, rel_tol=1e-14) and np.all(sig[1:] < 1e-12)
    assert np.allclose(np.abs(v[:, 0]), np.abs(y) / 5.0, atol=1e-14)


PINS = [pin_lapack_values, pin_orthonormal_and_reconstruction, pin_eckart_young, pin_hand_examples]


@pytest.mark.parametrize("pin", PINS, ids=lambda p: p.__name__)
def test_pin(pin):
    pin(oracle.block_svd)


MUTATIONS = [
    ("rotation sign flipped", "a[:, p], a[:, q] = c * ap - s_ * aq, s_ * ap + c * aq",
     "a[:, p], a[:, q] = c * ap + s_ * aq, -s_ * ap + c * aq"),
    ("V not rotated", "v[:, p], v[:, q] = c * vp - s_ * vq, s_ * vp + c * vq", "pass"),
    ("zeta halved", "zeta = (beta - alpha) / (2.0 * gamma)", "zeta = (beta - alpha) / (4.0 * gamma)"),
    ("squared values", "sigma = np.sqrt(np.sum(a * a, axis=0))", "sigma = np.sum(a * a, axis=0)"),
    ("ascending order", 'order = np.argsort(-sigma, kind="stable")', 'order = np.argsort(sigma, kind="stable")'),
    ("one sweep only", "        if not rotated:\n            break", "        break"),
]


@pytest.mark.parametrize("name,old,new", MUTATIONS, ids=[m[0] for m in MUTATIONS])
def test_planted_mistake_is_caught(name, old, new):
    src = inspect.getsource(oracle)
    assert src.count(old) == 1, f"mutation anchor not unique: {old!r}"
    ns = {"__name__": "oracle_mutant"}
    exec(compile(src.replace(old, new), "oracle_mutant", "exec"), ns)
    failed = []
    for pin in PINS:
        try:
            pin(ns["block_svd"])
        except Exception:
            failed.append(pin.__name__)
    assert failed, f"planted mistake '{name}' passed every pin"
