"""Pins for the oracle's INT8 storage of the P factors (per token row,
symmetric): exact recovery of rows that are a power-of-two scale times integer
codes, ties rounded to even, the half-step error bound and the full-scale code
at every row's largest magnitude, sign symmetry, zero rows, and the effect on
attention (a bounded perturbation).  Planted mistakes in a copy of the
quantiser (scale over 128, truncation, ties away from zero, per-column scales,
no clip) each fail a pin."""
import inspect

import numpy as np
import pytest

import oracle
from helpers import oracle_args
from synth import bf16_to_f32, make_problem


def pin_exact_rows(quant):
    """Rows s0 * c with s0 a power of two and integer codes reaching +-127
    quantise to exactly those codes and exactly that scale."""
    rng = np.random.default_rng(1)
    for s0 in (2.0 ** -7, 2.0 ** -2, 1.0, 8.0):
        c = rng.integers(-127, 128, size=(5, 9))
        c[:, 3] = np.where(rng.random(5) < 0.5, 127, -127)
        codes, scales = quant(s0 * c.astype(np.float32))
        assert np.array_equal(codes.astype(np.int64), c)
        assert np.array_equal(scales, np.full(5, s0, dtype=np.float32))


def pin_ties_to_even(quant):
    """Scale 1 (a row holding 127): values halfway between integers go to the
    even neighbour."""
    row = np.array([[127.0, 2.5, 3.5, -2.5, -3.5, 0.5, -0.5, 1.5, 126.5]], dtype=np.float32)
    codes, scales = quant(row)
    assert scales[0] == 1.0
    assert codes[0].tolist() == [127, 2, 4, -2, -4, 0, 0, 2, 126]


def pin_error_bound_and_full_scale(quant):
    """|P - s c| <= s / 2 (plus the rounding of the fp32 quotient), |c| <= 127,
    and each row's largest magnitude maps to +-127."""
    rng = np.random.default_rng(2)
    p = bf16_to_f32(np.frombuffer(rng.integers(0, 65535, 4000, dtype=np.uint16).tobytes(), np.uint16))
    p = p[np.isfinite(p)][:3000].reshape(-1, 30) * np.float32(1.0)
    codes, scales = quant(p)
    deq = scales[:, None].astype(np.float64) * codes
    assert np.all(np.abs(codes.astype(np.int64)) <= 127)
    assert np.all(np.abs(deq - p) <= scales[:, None].astype(np.float64) * (0.5 + 1e-6) + 1e-300)
    big = np.argmax(np.abs(p), axis=1)
    nz = scales > 0
    assert np.all(np.abs(codes[np.arange(len(p)), big].astype(np.int64))[nz] == 127)


def pin_sign_and_zero(quant):
    rng = np.random.default_rng(3)
    p = rng.standard_normal((6, 11)).astype(np.float32)
    p[2] = 0.0
    c1, s1 = quant(p)
    c2, s2 = quant(-p)
    assert np.array_equal(c1.astype(np.int64), -c2.astype(np.int64)) and np.array_equal(s1, s2)
    assert s1[2] == 0 and not np.any(c1[2])


PINS = [pin_exact_rows, pin_ties_to_even, pin_error_bound_and_full_scale, pin_sign_and_zero]


@pytest.mark.parametrize("pin", PINS, ids=lambda p: p.__name__)
def test_pin(pin):
    pin(oracle.quantize_rows_int8)


def test_dequantised_attention_stays_close():
    """Attention over INT8-stored P factors: the output moves by a small
    fraction of its norm (each P element moves by at most half a step, s / 2 =
    max|row| / 254)."""
    inp = make_problem(4, [300, 700, 64], [64, 160, 32], n_kv_heads=2, head_dim=64, n_q=3, n_q_heads=8,
                       tail_cap=20)
    a = oracle_args(inp)
    ref = oracle.attend_latent(**a)
    q = dict(a)
    q["pk"] = [oracle.dequantize_rows_int8(*oracle.quantize_rows_int8(p)) for p in a["pk"]]
    q["pv"] = [oracle.dequantize_rows_int8(*oracle.quantize_rows_int8(p)) for p in a["pv"]]
    got = oracle.attend_latent(**q)
    err = np.linalg.norm((got - ref).reshape(-1, 64), axis=1) / np.linalg.norm(ref.reshape(-1, 64), axis=1)
    print(f"INT8 P factors: output rel-L2 vs the bf16 factors, max {err.max():.2e}")
    assert err.max() < 2e-2


MUTATIONS = [
    ("scale over 128", "amax / np.float32(127.0)", "amax / np.float32(128.0)"),
    ("truncation", "q = np.rint(p[nz] / scales[nz, None])", "q = np.trunc(p[nz] / scales[nz, None])"),
    ("ties away from zero", "q = np.rint(p[nz] / scales[nz, None])",
     "q = np.sign(p[nz]) * np.floor(np.abs(p[nz] / scales[nz, None]) + 0.5)"),
    ("per-column scale", "amax = np.abs(p).max(axis=1) if", "amax = np.abs(p).max(axis=0)[:p.shape[0]] if"),
    ("no clip, codes wrap", "codes[nz] = np.clip(q, -127, 127).astype(np.int8)",
     "codes[nz] = (q * 1.01).astype(np.int64).astype(np.int8)"),
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
            pin(ns["quantize_rows_int8"])
        except Exception:
            failed.append(pin.__name__)
    assert failed, f"planted mistake '{name}' passed every pin"
