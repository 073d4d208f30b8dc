"""Pre-RoPE keys (milo_cache_set_rope) on the GPU, through the C ABI, against the
CPU oracle's attention over rotated keys (oracle.attend_dense with key_pos and
rope_theta) on the same seeded inputs, at the latent parity bar (max over
(query, head) of the relative L2 error <= 1e-2).  Every selected block is then
rebuilt and its keys rotated to their positions before attention.

Covered: head dims 64 and 128 (the two key-tile arrangements of the
reconstruction kernel), ragged blocks, positions given per block (overlapping,
out of order, up to the int32 limit, where the fp64 angle reduction matters) or
by default one after another, block subsets, positions changed on one cache,
rotation switched off again, prefill, a 7B-shaped layer, and the refusals
(INT8 caches, the no-allocation entry point, bad arguments).  Each case also
checks that the oracle with every block moved by a single position is beyond
the bar, so the comparison can see a position error."""
import zlib

import numpy as np
import pytest

import oracle
import synth
from helpers import TOL_REL_L2, GpuLayer, max_rel_l2, oracle_args, to_device
from test_gpu_parity import SHAPES, _random_case

pytestmark = pytest.mark.gpu

THETA = 1e6
LIMIT = (1 << 31) - 1  # padded rows' positions stay below this


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_29913_amd import milo
    milo.lib()


def _check(got, inp, key_pos, table=None, tail_len=None, label="", moved_check=True):
    assert np.all(np.isfinite(got)), "unwritten or non-finite outputs"
    a = oracle_args(inp, table, tail_len)
    ref = oracle.attend_dense(**a, key_pos=key_pos, rope_theta=THETA)
    err = max_rel_l2(got, ref)
    # the same with every block one position later
    moved = [p + 1 for p in key_pos]
    off = max_rel_l2(got, oracle.attend_dense(**a, key_pos=moved, rope_theta=THETA))
    print(f"[rope] {label}: max rel-L2 = {err:.3e} (blocks moved by one position: {off:.3e})", flush=True)
    assert err <= TOL_REL_L2
    if moved_check:
        assert off > 3 * TOL_REL_L2


def _positions(inp, seed):
    """Random first-token positions with each block's padded rows below 2^31 - 1."""
    rng = np.random.default_rng(seed)
    return [int(rng.integers(0, LIMIT - 256 * -(-int(t) // 256) + 1)) for t in inp.block_tokens]


@pytest.mark.parametrize("name", ["ragged_d128_g4", "d64_g7_two_col_tiles", "g16", "q7b_shape_5_blocks"])
def test_rope_every_block(name):
    from paper_2609_29913_amd import milo
    inp = synth.make_problem(zlib.crc32(name.encode()) % 1000, **SHAPES[name])
    key_pos = _positions(inp, 1)
    gl = GpuLayer(inp)
    try:
        milo.milo_cache_set_rope(gl.cache, THETA, key_pos)
        got = gl.attend().cpu().numpy()
        assert milo.milo_cache_recon_blocks(gl.cache) == inp.n_blocks
    finally:
        gl.free()
    _check(got, inp, key_pos, label=name)


@pytest.mark.parametrize("seed", range(6))
def test_rope_random_shapes(seed):
    """The parity suite's random problems (head dims, groups, ragged blocks and
    ranks up to 1024, subsets in any order, empty or ragged tails) with random
    positions; tiny or tail-dominated cases are not asked to show the
    one-position shift."""
    from paper_2609_29913_amd import milo
    inp, table = _random_case(seed)
    key_pos = _positions(inp, 100 + seed)
    gl = GpuLayer(inp)
    try:
        milo.milo_cache_set_rope(gl.cache, THETA, key_pos)
        got = gl.attend(table=table).cpu().numpy()
        assert milo.milo_cache_recon_blocks(gl.cache) == len(table)
    finally:
        gl.free()
    _check(got, inp, key_pos, table=table, label=f"random seed {seed}", moved_check=False)


def test_rope_default_positions_subsets_and_changes():
    """Default positions (blocks one after another in id order), a subset in
    another order, then new positions on the same cache (the plan is rebuilt),
    then the rotation switched off (the latent route again, bitwise as a fresh
    cache)."""
    from paper_2609_29913_amd import milo
    inp = synth.make_problem(23, [700, 1024, 100, 513], [64, 288, 32, 128], [96, 256, 16, 128], n_kv_heads=4,
                             head_dim=128, n_q=3, n_q_heads=28, tail_cap=90, tail_len=[90, 0, 45])
    default_pos = list(np.concatenate([[0], np.cumsum(inp.block_tokens)[:-1]]).astype(int))
    gl = GpuLayer(inp)
    try:
        milo.milo_cache_set_path(gl.cache, milo.MILO_PATH_LATENT)
        plain = gl.attend().cpu().numpy()
        milo.milo_cache_set_rope(gl.cache, THETA)
        _check(gl.attend().cpu().numpy(), inp, default_pos, label="default positions")
        table = [3, 1]
        _check(gl.attend(table=table).cpu().numpy(), inp, default_pos, table=table, label="subset [3, 1]")
        assert milo.milo_cache_recon_blocks(gl.cache) == 2
        new_pos = [2_000_000_000, 0, 77, 1_000_003]
        milo.milo_cache_set_rope(gl.cache, THETA, new_pos)
        _check(gl.attend(table=table).cpu().numpy(), inp, new_pos, table=table, label="new positions")
        # AUTO would keep these low-rank blocks latent; pre-RoPE keys are rebuilt all the same
        milo.milo_cache_set_path(gl.cache, milo.MILO_PATH_AUTO)
        _check(gl.attend().cpu().numpy(), inp, new_pos, label="new positions, AUTO path")
        assert milo.milo_cache_recon_blocks(gl.cache) == inp.n_blocks
        milo.milo_cache_set_path(gl.cache, milo.MILO_PATH_LATENT)
        milo.milo_cache_set_rope(gl.cache, 0.0)
        again = gl.attend().cpu().numpy()
        assert milo.milo_cache_recon_blocks(gl.cache) == 0
    finally:
        gl.free()
    assert np.array_equal(plain, again)
    assert max_rel_l2(again, oracle.attend_latent(**oracle_args(inp))) <= TOL_REL_L2


def test_rope_prefill():
    import torch
    from paper_2609_29913_amd import milo
    n_tok, tail_base = 160, 100
    inp = synth.make_problem(29, [1024, 300], [288, 64], n_kv_heads=4, head_dim=128, n_q=n_tok, n_q_heads=28,
                             tail_cap=tail_base + n_tok)
    key_pos = [40_000, 1_500]
    table = [0, 1]
    gl = GpuLayer(inp)
    try:
        milo.milo_cache_set_rope(gl.cache, THETA, key_pos)
        tk, tv = to_device(inp.tail_k[0]), to_device(inp.tail_v[0])
        out = torch.full(inp.q.shape, float("nan"), dtype=torch.float32, device="cuda")
        milo.milo_attend_prefill(gl.cache, table, gl.q, tk, tv, tail_base, inp.scale, out)
        torch.cuda.synchronize()
        got = out.cpu().numpy()
    finally:
        gl.free()
    a = oracle_args(inp, table)
    ref = oracle.attend_prefill(a["pk"], a["rk"], a["pv"], a["rv"], table, a["q"], a["tail_k"][0], a["tail_v"][0],
                                tail_base, inp.scale, key_pos=key_pos, rope_theta=THETA)
    err = max_rel_l2(got, ref)
    print(f"[rope] prefill 160 tokens: max rel-L2 = {err:.3e}", flush=True)
    assert err <= TOL_REL_L2


@pytest.mark.timeout(600)
def test_rope_7b_shaped_layer():
    """A whole 7B-shaped layer (64 blocks of 1024 tokens, ranks 64..512, 8
    queries x 28 heads, 256-token tails), blocks at their default positions
    (65,536 tokens), every column checked."""
    from paper_2609_29913_amd import milo
    inp = synth.gen_layer("q7b_1l", 0)
    key_pos = [1024 * b for b in range(inp.n_blocks)]
    gl = GpuLayer(inp)
    try:
        milo.milo_cache_set_rope(gl.cache, THETA)
        got = gl.attend().cpu().numpy()
    finally:
        gl.free()
    _check(got, inp, key_pos, label="q7b layer 0")


def test_rope_refusals():
    import torch
    from paper_2609_29913_amd import milo
    inp = synth.make_problem(5, [256, 100], [32, 64], n_kv_heads=1, head_dim=64, n_q=2, n_q_heads=2, tail_cap=4)
    gl = GpuLayer(inp)
    try:
        for theta in (1.0, -5.0, float("inf"), float("nan")):
            with pytest.raises(milo.MiloError, match="theta"):
                milo.milo_cache_set_rope(gl.cache, theta)
        for pos in ([-1, 0], [0, LIMIT - 255], [LIMIT - 255, 0]):
            with pytest.raises(milo.MiloError, match="must lie in"):
                milo.milo_cache_set_rope(gl.cache, THETA, pos)
        with pytest.raises(ValueError):
            milo.milo_cache_set_rope(gl.cache, THETA, [0])
        # the last valid position of a 100-token block padded to 256 rows
        milo.milo_cache_set_rope(gl.cache, THETA, [0, LIMIT - 256])
        out = torch.zeros(inp.q.shape, dtype=torch.float32, device="cuda")
        with pytest.raises(milo.MiloError, match="latent only"):
            milo.milo_attend_decode_noalloc(gl.cache, [0, 1], gl.q, gl.tk, gl.tv, inp.tail_len, inp.scale, out)
        _check(gl.attend().cpu().numpy(), inp, [0, LIMIT - 256], label="positions at the limit")
    finally:
        gl.free()
    g8 = GpuLayer(inp, p_int8=True)
    try:
        with pytest.raises(milo.MiloError, match="INT8"):
            milo.milo_cache_set_rope(g8.cache, THETA)
    finally:
        g8.free()
