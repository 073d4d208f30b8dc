"""The attention work plan (host logic, no GPU): built by the library's own
planner source for the benchmark workloads and random shapes, then decoded and
checked for exact coverage of every (block tile, column tile) pair and every
planned tail chunk, consistent partial slots and programs that fit in LDS
(tests/plan_check.cpp)."""
import os
import subprocess

import numpy as np
import pytest

import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2609_29913_amd", "csrc")


@pytest.fixture(scope="module")
def checker(tmp_path_factory):
    exe = str(tmp_path_factory.mktemp("plan") / "plan_check")
    cmd = ["g++", "-O2", "-std=c++17", "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include", "-I", CSRC,
           os.path.join(ROOT, "tests", "plan_check.cpp"), os.path.join(CSRC, "milo_plan.cpp"), "-o", exe]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        pytest.fail("could not build the plan checker:\n" + res.stderr[-3000:])
    return exe


def _case(n_kv, d, G, n_q, n_chunks, T, rk, rv=None, table=None, cap=-1, i8=False, recon=0, gemv=False):
    """recon: 0 every block latent, 1 every selected block reconstructed, 2 every
    other one; gemv: the projection runs as a GEMV (tiles of at most 16 columns)."""
    rv = rk if rv is None else rv
    table = list(range(len(T))) if table is None else table
    head = f"{n_kv} {d} {G} {n_q} {n_chunks} {cap} {int(i8)} {recon} {int(gemv)} {len(T)}"
    blocks = " ".join(f"{t} {a} {b}" for t, a, b in zip(T, rk, rv))
    return f"{head} {blocks} {len(table)} {' '.join(map(str, table))}\n"


def _run(checker, cases):
    res = subprocess.run([checker], input="".join(cases), capture_output=True, text=True)
    assert res.returncode == 0 and "OK" in res.stdout.splitlines()[-1], res.stdout[-4000:] + res.stderr
    return res.stdout


def _chunks(tail, cap):
    """Planned tail chunks: the longest tail rounded up to a power of two of
    256-token chunks, at most the tail buffer's chunks."""
    need = -(-tail // 256)
    if need == 0:
        return 0
    p = 1
    while p < need:
        p *= 2
    return min(p, -(-cap // 256))


def test_plans_of_the_workloads(checker):
    cases = []
    for name, cfg in synth.CONFIGS.items():
        T = synth.draw_block_tokens(cfg)
        for layer in (0, cfg.n_layers - 1):
            r = synth.draw_ranks(cfg, layer, len(T))
            cases.append(_case(cfg.n_kv_heads, cfg.head_dim, cfg.group, cfg.n_q, _chunks(cfg.tail, cfg.tail),
                               T, r))
    out = _run(checker, cases)
    print(out)


def test_plans_of_random_shapes(checker):
    rng = np.random.default_rng(7)
    cases = []
    for _ in range(60):
        d = int(rng.choice([64, 128]))
        n_kv = int(rng.choice([1, 2, 3, 4, 8]))
        G = int(rng.choice([1, 2, 5, 7, 16]))
        n_q = int(rng.integers(1, 70))
        nb = int(rng.integers(1, 40))
        T = rng.integers(1, 5000, nb)
        D = n_kv * d
        rk = [int(rng.integers(1, min(int(t), D, 896) + 1)) for t in T]
        rv = [int(rng.integers(1, min(int(t), D, 896) + 1)) for t in T]
        k = int(rng.integers(1, nb + 1))
        table = [int(b) for b in rng.permutation(nb)[:k]]
        cases.append(_case(n_kv, d, G, n_q, int(rng.integers(0, 5)), T, rk, rv, table, i8=bool(rng.integers(2))))
    _run(checker, cases)


def test_plan_split_over_launches(checker):
    """A program cap small enough to need several launches (1200 one-tile
    blocks on one KV head), and tail chunks with leftover solo workgroups."""
    n = 1200
    cases = [_case(1, 64, 2, 2, 1, [32] * n, [16] * n, [8] * n, cap=1792),
             _case(8, 128, 5, 16, 8, [1024] * 30, [320] * 30, cap=12000)]
    out = _run(checker, cases)
    assert "launches 1 " not in out.splitlines()[0]


def test_column_tiling_choices(checker):
    """Heads with few columns are packed into one tile; a 32B-shaped batch (80
    columns per KV head) uses ten head-spanning tiles instead of sixteen; the
    7B 28-layer and 14B batches keep per-head tiles."""
    cases = [_case(2, 64, 7, 1, 1, [512] * 8, [64] * 8),       # tiny: 14 columns, one tile
             _case(8, 128, 5, 16, 8, [1024] * 8, [320] * 8),   # 32B: 640 columns
             _case(4, 128, 7, 32, 2, [1024] * 8, [128] * 8),   # 7B 28 layers: 896 columns
             _case(8, 128, 5, 64, 4, [1024] * 8, [448] * 8)]   # 14B: 2560 columns
    lines = _run(checker, cases).splitlines()
    assert "tiles 1 (mode 0)" in lines[0]
    assert "tiles 10 (mode 2) gang 10" in lines[1]
    assert "tiles 16 (mode 1) gang 16" in lines[2]
    assert "tiles 40 (mode 1) gang 8" in lines[3]


def test_folded_slots_per_column_group(checker):
    """The 14B-shaped batch has five column groups per gang.  With every block
    rebuilt (dense items, foldable) each gang's items go by column group and fold
    into one slot per gang and tile: 32 slots per column tile instead of one per
    block.  The latent plan (ranks to 768, three rank tiles per wave: the kernel
    does not fold) keeps one slot per block and its order by length."""
    cfg = synth.CONFIGS["q14b_48l"]
    T = synth.draw_block_tokens(cfg)
    r = synth.draw_ranks(cfg, 0, len(T))
    args = (cfg.n_kv_heads, cfg.head_dim, cfg.group, cfg.n_q, _chunks(cfg.tail, cfg.tail), T, r)
    lines = _run(checker, [_case(*args, recon=1), _case(*args, recon=0)]).splitlines()
    assert "gang 8" in lines[0] and "slots 32 " in lines[0], lines[0]
    assert "slots 256 " in lines[1], lines[1]


def test_plans_with_reconstructed_blocks(checker):
    """Reconstruct-then-attend plans: every block or every other block rebuilt,
    on the workloads and on random shapes (few and many columns per KV head):
    dense items per head tile, reconstruction tasks covering each (block, side,
    head, tile) once with each block side on one XCD."""
    cases = []
    for name, cfg in synth.CONFIGS.items():
        T = synth.draw_block_tokens(cfg)
        r = synth.draw_ranks(cfg, 0, len(T))
        for mode in (1, 2):
            cases.append(_case(cfg.n_kv_heads, cfg.head_dim, cfg.group, cfg.n_q, _chunks(cfg.tail, cfg.tail), T, r,
                               recon=mode))
    rng = np.random.default_rng(11)
    for _ in range(40):
        d = int(rng.choice([64, 128]))
        n_kv = int(rng.choice([1, 2, 3, 4, 8]))
        G = int(rng.choice([1, 2, 5, 7, 16]))
        n_q = int(rng.integers(1, 70))
        nb = int(rng.integers(1, 30))
        T = rng.integers(1, 5000, nb)
        D = n_kv * d
        rk = [int(rng.integers(1, min(int(t), D, 896) + 1)) for t in T]
        rv = [int(rng.integers(1, min(int(t), D, 896) + 1)) for t in T]
        k = int(rng.integers(1, nb + 1))
        table = [int(b) for b in rng.permutation(nb)[:k]]
        cases.append(_case(n_kv, d, G, n_q, int(rng.integers(0, 5)), T, rk, rv, table, recon=int(rng.integers(1, 3))))
    _run(checker, cases)


def test_gemv_tiling(checker):
    """With the GEMV projection, tiles that pack whole KV heads hold at most 16
    columns: 7 columns per head -> two heads per tile, 2 -> four, 16 -> one; the
    MFMA projection packs up to 64."""
    cases = [_case(8, 128, 7, 1, 1, [512] * 4, [64] * 4, gemv=True),
             _case(8, 64, 2, 1, 1, [512] * 4, [64] * 4, gemv=True),
             _case(4, 128, 4, 4, 1, [512] * 4, [64] * 4, gemv=True),
             _case(8, 128, 7, 1, 1, [512] * 4, [64] * 4, gemv=False)]
    lines = _run(checker, cases).splitlines()
    assert "tiles 4 (mode 0)" in lines[0]
    assert "tiles 2 (mode 0)" in lines[1]
    assert "tiles 4 (mode 0)" in lines[2]
    assert "tiles 2 (mode 0)" in lines[3]
