"""The encoder's per-block truncated SVD on the GPU (milo_block_svd /
milo_block_factors, through the C ABI) against the oracle's one-sided Jacobi
SVD (fp64) on the same bf16 blocks, by properties that hold at any size on a
full 7B-shaped block, and end to end: blocks -> singular values -> entropy
rank allocation -> factors -> cache -> decode, checked against the oracle on
the factors the GPU produced."""
import numpy as np
import pytest

import oracle
import synth
from helpers import TOL_REL_L2, GpuLayer, max_rel_l2, oracle_args

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_29913_amd import milo
    milo.lib()


def _dev(a):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).cuda()


def _f64(a):
    return synth.bf16_to_f64(a)


# (T, D, decay): square, tall, wide (T < D, only T non-zero values), odd D (padded to even),
# a D that is not a multiple of the 64-wide Gram tiles, a flat spectrum
SHAPES = [(64, 64, 0.8), (300, 128, 1.0), (40, 128, 0.6), (129, 65, 0.9), (200, 96, 0.7), (128, 128, 0.1)]


def test_singular_values_and_vectors_match_the_oracle():
    from paper_2609_29913_amd import milo
    blocks = [synth.gen_kv_block(i, T, D, dec) for i, (T, D, dec) in enumerate(SHAPES)]
    for blk, (T, D, _) in zip(blocks, SHAPES):
        sigma, vt = milo.milo_block_svd([_dev(blk)])
        sg, vg = sigma[0].cpu().numpy().astype(np.float64), vt[0].cpu().numpy().astype(np.float64)
        sr, vr = oracle.block_svd(_f64(blk))
        lam_g, lam_r = sg ** 2, sr ** 2
        # eigenvalues of the fp32 Gram matrix: absolute error ~ eps * lambda_max
        err = np.abs(lam_g - lam_r)
        print(f"[svd] T={T} D={D}: max |lambda_gpu - lambda_ref| / lambda_max = {err.max() / lam_r[0]:.2e}, "
              f"{milo.milo_block_svd_sweeps()} sweeps", flush=True)
        assert np.all(err <= 1e-5 * lam_r[0] + 1e-3 * lam_r)
        assert milo.milo_block_svd_sweeps() < 30
        assert np.all(np.diff(sg) <= 1e-6 * sg[0])
        # vectors: unit norm, orthogonal, and along the oracle's where the spectrum separates them
        assert np.allclose(vg @ vg.T, np.eye(D), atol=2e-4)
        n = min(T, D)
        for j in range(n):
            gap = min(sr[j - 1] - sr[j] if j else np.inf, sr[j] - sr[j + 1] if j + 1 < n else np.inf)
            if gap > 0.05 * sr[0] and sr[j] > 0.05 * sr[0]:
                assert abs(vg[j] @ vr[:, j]) > 1 - 1e-3, (T, D, j)


def test_full_block_by_properties():
    """A 7B-shaped block (1024 tokens, D = 512): non-increasing values, the
    squares summing to ||K||_F^2, orthonormal V, and ||K v_j|| = sigma_j for
    the leading 32."""
    from paper_2609_29913_amd import milo
    blk = synth.gen_kv_block(40, 1024, 512, 0.9)
    sigma, vt = milo.milo_block_svd([_dev(blk)])
    sg, vg = sigma[0].cpu().numpy().astype(np.float64), vt[0].cpu().numpy().astype(np.float64)
    k = _f64(blk)
    print(f"[svd] 1024 x 512 block: {milo.milo_block_svd_sweeps()} Jacobi sweeps", flush=True)
    assert milo.milo_block_svd_sweeps() < 30
    assert np.all(np.diff(sg) <= 1e-6 * sg[0])
    assert abs(np.sum(sg ** 2) / np.sum(k * k) - 1) < 1e-4
    assert np.abs(vg @ vg.T - np.eye(512)).max() < 2e-4
    kv = np.linalg.norm(k @ vg[:32].T, axis=0)
    assert np.allclose(kv, sg[:32], rtol=1e-3)


def test_factors_reach_the_eckart_young_error():
    """||K - P R||_F of the bf16 factors at rank r is the optimum
    sqrt(sum_{j>r} sigma_j^2) (oracle, fp64) plus the bf16 rounding of P and R."""
    from paper_2609_29913_amd import milo
    # three blocks of one width per call, of different lengths and ranks
    for i, (T, D, dec) in enumerate(SHAPES[:4]):
        blocks = [synth.gen_kv_block(50 + 3 * i + j, T - 17 * j, D, dec) for j in range(3)]
        dev = [_dev(b) for b in blocks]
        sigma, vt = milo.milo_block_svd(dev)
        ranks = [max(1, min(T - 17 * j, D) // (3 + j)) for j in range(3)]
        ps, rs = milo.milo_block_factors(dev, vt, ranks)
        _check_factors(blocks, ps, rs, ranks)


def _check_factors(blocks, ps, rs, ranks):
    for blk, p, r, rank in zip(blocks, ps, rs, ranks):
        k = _f64(blk)
        pr = synth.bf16_to_f64(p.cpu().numpy().view(np.uint16)) @ synth.bf16_to_f64(r.cpu().numpy().view(np.uint16))
        sr, _ = oracle.block_svd(k)
        opt = np.sqrt(np.sum(sr[rank:] ** 2))
        got = np.linalg.norm(k - pr)
        print(f"[svd] rank {rank}: ||K - P R|| = {got:.4e}, optimum {opt:.4e}, ||K|| = {np.linalg.norm(k):.4e}",
              flush=True)
        assert got <= opt + 4e-3 * np.linalg.norm(k)


def test_encoder_pipeline_feeds_the_decode_step():
    """Keys and values of 4 blocks -> GPU SVD -> entropy rank allocation (keys
    and values apart, half the full-rank budget) -> GPU factors -> cache ->
    decode step, checked against the oracle on the factors the GPU produced;
    the distance to dense attention over the original keys and values is the
    compression error (reported)."""
    import torch
    from paper_2609_29913_amd import milo
    n_kv, d, G, n_q = 2, 64, 4, 3
    D = n_kv * d
    T = [512, 300, 256, 100]
    K = [synth.gen_kv_block(60 + b, t, D, 1.0) for b, t in enumerate(T)]
    V = [synth.gen_kv_block(70 + b, t, D, 0.7) for b, t in enumerate(T)]
    kd, vd = [_dev(x) for x in K], [_dev(x) for x in V]
    n_sv = [min(t, D) for t in T]
    budget = sum(n_sv) // 2
    ranks = {}
    facs = {}
    for name, dev in (("k", kd), ("v", vd)):
        sigma, vt = milo.milo_block_svd(dev)
        r = milo.milo_allocate_ranks(sigma, n_sv, budget, 8, D)
        ranks[name] = r
        facs[name] = milo.milo_block_factors(dev, vt, r)
    pk, rk = [p.cpu().numpy().view(np.uint16) for p in facs["k"][0]], [x.cpu().numpy().view(np.uint16) for x in facs["k"][1]]
    pv, rv = [p.cpu().numpy().view(np.uint16) for p in facs["v"][0]], [x.cpu().numpy().view(np.uint16) for x in facs["v"][1]]
    rng = np.random.default_rng(80)
    inp = synth.LayerInputs(n_kv_heads=n_kv, head_dim=d, n_q_heads=n_kv * G, block_tokens=np.array(T, np.int32),
                            rank_k=np.array(ranks["k"], np.int32), rank_v=np.array(ranks["v"], np.int32),
                            pk=pk, rk=rk, pv=pv, rv=rv,
                            q=synth.f32_to_bf16(rng.standard_normal((n_q, n_kv * G, d)).astype(np.float32)),
                            tail_k=synth.f32_to_bf16(rng.standard_normal((n_q, 16, n_kv, d)).astype(np.float32)),
                            tail_v=synth.f32_to_bf16(rng.standard_normal((n_q, 16, n_kv, d)).astype(np.float32)),
                            tail_len=np.array([16, 3, 0], np.int32), scale=1.0 / np.sqrt(d))
    gl = GpuLayer(inp)
    try:
        got = gl.attend().cpu().numpy()
    finally:
        gl.free()
    a = oracle_args(inp)
    err = max_rel_l2(got, oracle.attend_latent(**a))
    # compression error: dense attention over the original blocks (P = K, R = I)
    dense = dict(a, pk=[_f64(x) for x in K], rk=[np.eye(D)] * 4, pv=[_f64(x) for x in V], rv=[np.eye(D)] * 4)
    comp = max_rel_l2(got, oracle.attend_dense(**dense))
    print(f"[svd] pipeline: ranks K {ranks['k'].tolist()} V {ranks['v'].tolist()}; decode vs oracle on the GPU factors "
          f"{err:.3e}; vs dense attention on the original blocks {comp:.3e}", flush=True)
    assert err <= TOL_REL_L2
    assert sum(ranks["k"]) <= budget and sum(ranks["v"]) <= budget
