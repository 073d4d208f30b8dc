"""Packed factor layout (host logic, no GPU): the fragment order the kernels
stream must be a bijection onto the padded source block for every factor, and
the fragment index helpers (used by the reconstruction kernel) its inverse."""
import os
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
GEOMS = [
    (1, 1, 1, 64), (45, 33, 3, 64), (256, 64, 2, 128), (300, 100, 4, 128), (1024, 288, 4, 128),
    (700, 96, 2, 64), (1000, 896, 8, 128), (2048, 512, 8, 128), (513, 160, 1, 64), (100, 40, 4, 128),
    # every split of the latent value pass (1, 2, 4 and 8 token segments)
    (256, 32, 2, 64), (512, 64, 2, 64), (300, 96, 4, 128), (256, 128, 2, 64), (256, 224, 4, 128),
    (768, 288, 4, 128), (256, 384, 4, 128), (1024, 768, 8, 128),
]


@pytest.fixture(scope="module")
def checker(tmp_path_factory):
    exe = str(tmp_path_factory.mktemp("layout") / "layout_check")
    cmd = ["g++", "-O2", "-std=c++17", "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include",
           "-I", os.path.join(ROOT, "paper_2609_29913_amd", "csrc"),
           os.path.join(ROOT, "tests", "layout_check.cpp"), "-o", exe]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        pytest.fail("could not build the layout checker:\n" + res.stderr[-3000:])
    return exe


def test_fragment_layout_is_a_bijection(checker):
    args = [str(x) for g in GEOMS for x in g]
    res = subprocess.run([checker, *args], capture_output=True, text=True)
    assert res.returncode == 0, res.stdout + res.stderr
    assert res.stdout.startswith("OK")


# (T, rank_k, rank_v, KV heads, head dim): ragged tokens, K/V ranks that
# differ, every token-segment split of the value pass, ranks beyond 512
RUN_GEOMS = [
    (1, 1, 1, 1, 64), (45, 33, 17, 3, 64), (256, 64, 64, 2, 128), (300, 100, 257, 4, 128),
    (1024, 288, 288, 4, 128), (700, 96, 32, 2, 64), (1000, 896, 840, 8, 128), (2048, 512, 512, 8, 128),
    (513, 160, 224, 1, 64), (256, 32, 32, 2, 64), (512, 64, 128, 2, 64), (768, 288, 384, 4, 128),
    (1024, 768, 704, 8, 128),
]


def test_derived_fragment_runs_cover_each_block_once(checker):
    """The runs each wave derives for a block item (block_runs) read every
    P^K / P^V fragment once over the eight waves and every fragment of the
    item's head slices of R^K once and of R^V once per wave sharing its
    16-dim slice, with per-phase run lengths equal to what the kernel takes."""
    args = [str(x) for g in RUN_GEOMS for x in g]
    res = subprocess.run([checker, "--runs", *args], capture_output=True, text=True)
    assert res.returncode == 0, res.stdout + res.stderr
    assert res.stdout.startswith("OK")


def test_int8_runs_cover_codes_and_scales_once(checker):
    """INT8 P factors: the runs of the eight waves read every int8 fragment of
    P^K and P^V once, in whole 1 KiB units of two, and every (tile, wave) scale
    unit once, by its own wave, between its P^K and P^V runs."""
    args = [str(x) for g in RUN_GEOMS for x in g]
    res = subprocess.run([checker, "--runs-int8", *args], capture_output=True, text=True)
    assert res.returncode == 0, res.stdout + res.stderr
    assert res.stdout.startswith("OK")


def test_reconstructed_blocks_are_stored_and_read_once(checker):
    """Reconstruct-then-attend: the reconstruction kernel's packed stores put
    K_{b,g} and V_{b,g} exactly where the P^K / P^V layouts of rank d keep
    them, every fragment once, and a dense item's derived runs read each of
    them once (no R runs), for ragged token counts, 1..8 KV heads, d = 64 / 128."""
    geoms = [(1, 1, 64), (256, 2, 128), (300, 4, 128), (1000, 8, 128), (513, 3, 64), (2048, 8, 128), (45, 1, 128)]
    res = subprocess.run([checker, "--dense", *[str(x) for g in geoms for x in g]], capture_output=True, text=True)
    assert res.returncode == 0, res.stdout + res.stderr
    assert res.stdout.startswith("OK")
