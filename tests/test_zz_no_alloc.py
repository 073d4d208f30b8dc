"""The no-allocation entry point (milo_attend_decode_noalloc) against the
regular one (milo_attend_decode) through the C ABI: two calls in a row, the
second with a smaller input (fewer blocks, fewer queries, shorter tails), each
bitwise equal to the regular entry point's output and within the parity bar of
the oracle; a call whose workspace exceeds the scratch is refused before
anything is queued."""
import numpy as np
import pytest
import torch

import oracle
import synth
from helpers import TOL_REL_L2, GpuLayer, max_rel_l2, oracle_args, to_device

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_29913_amd import milo
    milo.lib()


def _both(gl, inp, table, q, tk, tv, tail_len):
    from paper_2609_29913_amd import milo
    a = torch.full(q.shape, float("nan"), dtype=torch.float32, device="cuda")
    b = torch.full(q.shape, float("nan"), dtype=torch.float32, device="cuda")
    milo.milo_attend_decode(gl.cache, table, q, tk, tv, tail_len, inp.scale, a)
    milo.milo_attend_decode_noalloc(gl.cache, table, q, tk, tv, tail_len, inp.scale, b)
    torch.cuda.synchronize()
    return a.cpu().numpy(), b.cpu().numpy()


def test_noalloc_matches_the_regular_entry_point_twice_then_smaller():
    inp = synth.make_problem(60, [1024, 700, 300, 2048], [288, 96, 64, 512], n_kv_heads=8, head_dim=128, n_q=16,
                             n_q_heads=40, tail_cap=300,
                             tail_len=[300, 0, 17, 256, 257, 1, 299, 100, 5, 300, 64, 128, 3, 9, 200, 77])
    gl = GpuLayer(inp)
    try:
        # call 1: the whole problem (ten head-spanning column tiles, two gangs' worth of parts)
        table = [0, 1, 2, 3]
        reg, noa = _both(gl, inp, table, gl.q, gl.tk, gl.tv, inp.tail_len)
        assert np.all(np.isfinite(noa))
        assert np.array_equal(reg.view(np.uint32), noa.view(np.uint32))
        err = max_rel_l2(noa, oracle.attend_latent(**oracle_args(inp, table)))
        print(f"[noalloc] call 1: bitwise equal to milo_attend_decode, rel-L2 vs oracle {err:.3e}", flush=True)
        assert err <= TOL_REL_L2
        # call 2: smaller (two blocks, 5 queries, shorter tails): a new plan in the same scratch
        n2 = 5
        q2 = to_device(inp.q[:n2])
        tk2 = to_device(np.ascontiguousarray(inp.tail_k[:n2]))
        tv2 = to_device(np.ascontiguousarray(inp.tail_v[:n2]))
        tl2 = [7, 0, 256, 1, 40]
        table2 = [2, 0]
        reg2, noa2 = _both(gl, inp, table2, q2, tk2, tv2, tl2)
        assert np.all(np.isfinite(noa2))
        assert np.array_equal(reg2.view(np.uint32), noa2.view(np.uint32))
        small = synth.LayerInputs(**{**inp.__dict__, "q": inp.q[:n2], "tail_k": inp.tail_k[:n2],
                                     "tail_v": inp.tail_v[:n2], "tail_len": np.array(tl2, dtype=np.int32)})
        err2 = max_rel_l2(noa2, oracle.attend_latent(**oracle_args(small, table2)))
        print(f"[noalloc] call 2 (smaller): bitwise equal, rel-L2 vs oracle {err2:.3e}", flush=True)
        assert err2 <= TOL_REL_L2
    finally:
        gl.free()


def test_noalloc_refuses_a_workspace_beyond_the_scratch():
    """2560 columns (64 queries x 40 heads) over 60 blocks of rank 544 (above
    512, where every block item writes its own partial): at least 60 partial
    slots per column tile, ~80 MB of partial results, beyond the 55 MiB region;
    the call is refused and the output keeps its fill."""
    from paper_2609_29913_amd import milo
    n = 60
    inp = synth.make_problem(61, [544] * n, [544] * n, n_kv_heads=8, head_dim=128, n_q=64, n_q_heads=40,
                             tail_cap=0)
    gl = GpuLayer(inp)
    try:
        out = torch.full(inp.q.shape, 3.0, dtype=torch.float32, device="cuda")
        with pytest.raises(milo.MiloError) as ei:
            milo.milo_attend_decode_noalloc(gl.cache, list(range(n)), gl.q, None, None, None, inp.scale, out)
        assert ei.value.code == milo.MILO_ERR_UNSUPPORTED and "scratch" in str(ei.value)
        torch.cuda.synchronize()
        assert bool((out == 3.0).all())
    finally:
        gl.free()
