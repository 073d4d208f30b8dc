"""The Python binding rejects misuse before anything reaches the library: host
arrays or CPU tensors where device buffers are required, wrong element types,
strided views, and shapes that disagree with the cache (head dim, KV heads,
request count, tail capacity).  The CPU tests need no GPU; the GPU-marked
ones build a small cache and check that each bad call raises ValueError and
queues nothing (the output keeps its fill)."""
import numpy as np
import pytest
import torch

import synth
from paper_2609_29913_amd import milo


def test_host_buffers_are_rejected_for_device_arguments():
    milo.lib()
    q = np.zeros((1, 4, 64), dtype=np.uint16)
    out = torch.zeros((1, 4, 64), dtype=torch.float32)
    for bad_q, bad_out in ((q, out), (torch.zeros((1, 4, 64), dtype=torch.int16), out)):
        with pytest.raises(ValueError):
            milo.milo_attend_decode(12345, [0], bad_q, None, None, None, 0.125, bad_out)
        with pytest.raises(ValueError):
            milo.milo_attend_prefill(12345, [0], bad_q, None, None, 0, 0.125, bad_out)


def test_sigma_must_be_a_float32_gpu_tensor():
    milo.lib()
    for sigma in (np.ones((2, 4), dtype=np.float32), torch.ones((2, 4), dtype=torch.float32)):
        with pytest.raises(ValueError):
            milo.milo_allocate_ranks(sigma, [4, 4], 4, 1, 4)


def test_create_checks_factor_shapes_and_types():
    milo.lib()
    inp = synth.make_problem(3, [64, 32], [8, 4], n_kv_heads=2, head_dim=64, n_q=1, n_q_heads=2)
    bad_shape = list(inp.rk)
    bad_shape[1] = bad_shape[1][:, :64]                       # R^K with d columns instead of H_kv * d
    bad_type = [x.astype(np.float32) for x in inp.pk]         # values, not bf16 bit patterns
    for pk, rk in ((inp.pk, bad_shape), (bad_type, inp.rk)):
        with pytest.raises(ValueError):
            milo.milo_cache_create(inp.block_tokens, inp.rank_k, inp.rank_v, 2, 64, pk, rk, inp.pv, inp.rv)
    with pytest.raises(ValueError):
        milo.milo_cache_create(inp.block_tokens[:1], inp.rank_k, inp.rank_v, 2, 64, inp.pk, inp.rk, inp.pv,
                               inp.rv)


@pytest.mark.gpu
def test_device_argument_mismatches_raise_before_queuing():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from helpers import GpuLayer
    inp = synth.make_problem(4, [64, 64], [16, 16], n_kv_heads=2, head_dim=64, n_q=2, n_q_heads=4, tail_cap=8)
    gl = GpuLayer(inp)
    try:
        out = torch.full(inp.q.shape, 7.0, dtype=torch.float32, device="cuda")
        good = dict(block_table=[0, 1], q=gl.q, tail_k=gl.tk, tail_v=gl.tv, tail_len=[8, 3], scale=inp.scale,
                    out=out)
        cases = [
            dict(q=gl.q.float()),                                   # fp32 query
            dict(q=gl.q[:, :, :32].contiguous()),                   # head dim 32 vs the cache's 64
            dict(q=gl.q.transpose(0, 1)),                           # strided view
            dict(out=out.double()),
            dict(out=out[:1]),                                      # shape differs from q
            dict(tail_k=gl.tk[:, :, :1].contiguous()),              # one KV head vs two
            dict(tail_v=None),
            dict(tail_k=gl.tk[:1], tail_v=gl.tv[:1]),               # tails for one request, two queries
            dict(tail_len=[8]),                                     # one length for two requests
        ]
        for kw in cases:
            args = dict(good)
            args.update(kw)
            with pytest.raises(ValueError):
                milo.milo_attend_decode(gl.cache, **args)
        with pytest.raises(ValueError):
            milo.milo_attend_decode(gl.cache + 8, **good)          # not a handle this process made
        torch.cuda.synchronize()
        assert bool((out == 7.0).all()), "a rejected call wrote the output"
        with pytest.raises(ValueError):
            milo.milo_attend_prefill(gl.cache, [0], gl.q, gl.tk, gl.tv, 0, inp.scale, out)  # 4-D tail
    finally:
        gl.free()
