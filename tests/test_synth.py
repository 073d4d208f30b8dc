"""Seeded input generator: determinism, distributions, rank sets, block sizes."""
import numpy as np
import pytest

import synth
from synth import CONFIGS, bf16_to_f32, draw_block_tokens, draw_ranks, f32_to_bf16, gen_layer


def test_bf16_round_to_nearest_even():
    x = np.array([1.0, 1.0 + 2**-8, 1.0 + 3 * 2**-8, 1.0 + 2**-9, -2.5, 3.0e38], dtype=np.float32)
    got = bf16_to_f32(f32_to_bf16(x))
    # 1+2^-8 is a tie between 1 and 1+2^-7 -> even (1.0); 1+3*2^-8 ties up to 1+2^-6
    assert got[0] == 1.0 and got[1] == 1.0 and got[2] == np.float32(1.0 + 2**-6)
    assert got[3] == 1.0 and got[4] == -2.5
    assert np.isclose(got[5], 3.0e38, rtol=2**-8)


def test_tiny_is_deterministic():
    a, b = gen_layer("tiny"), gen_layer("tiny")
    for x, y in zip(a.pk + a.rv + [a.q, a.tail_k], b.pk + b.rv + [b.q, b.tail_k]):
        assert np.array_equal(x, y)
    c = gen_layer("tiny", layer=1)
    assert not np.array_equal(a.pk[0][:4], c.pk[0][:4]) or not np.array_equal(a.rank_k, c.rank_k)


def test_tiny_shapes_and_moments():
    inp = gen_layer("tiny")
    assert inp.n_blocks == 8 and set(inp.rank_k.tolist()) <= {32, 64, 96, 128}
    assert inp.q.shape == (1, 14, 64) and inp.tail_k.shape == (1, 64, 2, 64)
    p = np.concatenate([bf16_to_f32(x).ravel() for x in inp.pk])
    assert abs(p.mean()) < 0.01 and abs(p.var() - 1.0) < 0.02
    for r, rk in zip(inp.rank_k, inp.rk):
        v = bf16_to_f32(rk).var()
        assert abs(v * r - 1.0) < 0.05
    assert inp.scale == pytest.approx(1 / 8)


@pytest.mark.parametrize("name", list(CONFIGS))
def test_rank_sets(name):
    cfg = CONFIGS[name]
    bt = draw_block_tokens(cfg)
    assert int(bt.sum()) == cfg.context
    for layer in (0, cfg.n_layers - 1):
        r = draw_ranks(cfg, layer, len(bt))
        assert np.all(r <= np.minimum(bt, cfg.d_kv)) and np.all(r % 32 == 0)
        if name == "q7b_1l":
            assert set(r.tolist()) <= set(range(64, 513, 32))
        if name == "q7b_28l":
            hi = r >= 384
            assert hi.sum() == round(0.2 * len(bt))
            assert set(r[~hi].tolist()) <= {64, 96, 128, 160}
        if name == "q14b_48l":
            assert set(r.tolist()) <= set(range(128, 769, 64))
        if name == "q32b_64l":
            assert set(r.tolist()) <= set(range(128, 513, 32))
            assert set(bt.tolist()) <= {512, 1024, 2048}


def test_accounting_tiny():
    inp = gen_layer("tiny")
    D = 128
    fac = sum(2 * (512 + D) * 2 * int(r) for r in inp.rank_k)
    assert synth.algorithmic_bytes(inp) == fac + 4 * 64 * D + 6 * 14 * 64
