#!/usr/bin/env python3
"""Decode-step benchmark: low-rank (block-wise factorised) KV-cache attention on one GPU.

One step = one milo_attend_decode per layer of the workload: latent query
projection, scores + online softmax + latent V, up-projection, dense tail and
the log-sum-exp merge, for every query column of the decode batch.  Inputs are
seeded synthetic tensors with the workload's shapes, resident in HBM before the
timed region.  The default workload is the largest that fits one GPU: a
Qwen2.5-32B-shaped step of 64 layers (40 query / 8 KV heads, d=128, 1,048,576
context tokens in ragged blocks of 512/1024/2048, ranks 128..512, 2048-token
dense tail per request, 16 decode queries; ~170 GB of factors in HBM).  Other
workloads via --config; a single-layer working set (e.g. the 7B-shaped layer,
~117 MB) fits in the 256 MB Infinity Cache, so its steps rotate over
independent copies of the layer (each with its own cache, queries and tails)
until the rotation exceeds 512 MB.

Prints one JSON line (see the fields below).  --gpus above 1 is rejected: this
path runs on one GPU.  --prefill N measures instead the causal prefill of one
request's chunk of N tokens (milo_attend_prefill) on the workload's first layer,
after the workload's tail length of earlier tokens, and prints one JSON line for it.
--alloc measures instead the encoder's entropy rank allocation (milo_allocate_ranks)
on one layer's synthetic key spectra with the workload's block sizes.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import synth  # noqa: E402

METRIC = "effective context tokens/s per decode step (1 GPU) + % of HBM roofline"
HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, AMD published
MFMA_BF16_PEAK_TFLOPS = 2500.0  # MI355X dense bf16 MFMA, AMD published
KERNEL_SOURCES = [os.path.join(ROOT, "paper_2609_29913_amd", "csrc", f)
                  for f in ("milo_kernels.hip", "milo_internal.h", "milo_api.cpp", "milo_plan.cpp", "milo_plan.h")]


ALLOC_SOURCES = [os.path.join(ROOT, "paper_2609_29913_amd", "csrc", f) for f in ("milo_alloc.hip", "milo_alloc.h")]


def kernel_source_hash(sources=None) -> str:
    h = hashlib.sha256()
    for p in (KERNEL_SOURCES if sources is None else sources):
        with open(p, "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def counter_summary(workload: str) -> str:
    return os.path.join(ROOT, "profiles", f"attend_kernel_{workload}_counters.md")


def workload_name(cfg, args) -> str:
    """The workload as the JSON line and the profile summaries name it."""
    path = getattr(args, "path", "latent")
    rope = getattr(args, "rope", 0.0) > 0
    return (cfg.name + ("_int8" if getattr(args, "int8", False) else "") +
            ("_rope" if rope else "" if path == "latent" else f"_{path}"))


PATHS = {"latent": 0, "reconstruct": 1, "auto": 2}  # MILO_PATH_* of milo_cache_set_path


def counter_values(workload: str):
    """(HBM bytes per attention-kernel launch, MFMA busy fraction) from the
    committed rocprofv3 counter summary of this workload, or (None, None) when
    absent or taken on different kernel sources."""
    path = counter_summary(workload)
    if not os.path.exists(path):
        return None, None
    txt = open(path).read()
    m = re.search(r"traffic_bytes_per_launch:\s*([0-9.eE+]+)", txt)
    busy = re.search(r"mfma_busy_frac:\s*([0-9.eE+]+)", txt)
    hsh = re.search(r"kernel_source_sha256_16:\s*([0-9a-f]+)", txt)
    if not m or not hsh or hsh.group(1) != kernel_source_hash():
        return None, None
    return float(m.group(1)), (float(busy.group(1)) if busy else None)


def to_device(a, dev):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to(dev)


class Layer:
    """One layer's device state: its cache, queries, tails and output (the host
    copies of the factors are not kept)."""

    def __init__(self, inp: synth.LayerInputs, dev, p_int8: bool = False, path: str = "latent", rope: float = 0.0):
        import torch
        from paper_2609_29913_amd import milo
        self.cache = milo.milo_cache_create(inp.block_tokens, inp.rank_k, inp.rank_v, inp.n_kv_heads,
                                            inp.head_dim, inp.pk, inp.rk, inp.pv, inp.rv, p_int8=p_int8)
        if path != "latent":
            milo.milo_cache_set_path(self.cache, PATHS[path])
        if rope > 0:
            milo.milo_cache_set_rope(self.cache, rope)  # blocks one after another from position 0
        self.q = to_device(inp.q, dev)
        self.tk = to_device(inp.tail_k, dev)
        self.tv = to_device(inp.tail_v, dev)
        self.out = torch.empty(inp.q.shape, dtype=torch.float32, device=dev)
        self.table = np.arange(inp.n_blocks, dtype=np.int32)
        self.tail_len = inp.tail_len.copy()
        self.tail_cap = inp.tail_cap
        self.scale = inp.scale

    def step(self, stream, grow: int = 0):
        """One decode call; grow > 0 lengthens every request's tail by that many
        tokens first (a decode loop appending each step's key and value)."""
        from paper_2609_29913_amd import milo
        if grow:
            self.tail_len = np.minimum(self.tail_len + grow, self.tail_cap)
        milo.milo_attend_decode(self.cache, self.table, self.q, self.tk, self.tv, self.tail_len, self.scale,
                                self.out, stream=stream)


class PrefillLayer(Layer):
    """A layer's cache plus one request's chunk of n_tok query tokens and its one
    shared tail (tail_base earlier rows, then the chunk's own rows)."""

    def __init__(self, inp: synth.LayerInputs, dev, n_tok: int, tail_base: int, seed: int):
        super().__init__(inp, dev)
        import torch
        rng = np.random.Generator(np.random.Philox(key=[0x50524546, seed]))
        D = inp.n_kv_heads * inp.head_dim
        q = synth.f32_to_bf16(rng.standard_normal((n_tok, inp.n_q_heads, inp.head_dim), dtype=np.float32))
        rows = tail_base + n_tok
        tk = synth.f32_to_bf16(rng.standard_normal((rows, inp.n_kv_heads, inp.head_dim), dtype=np.float32))
        tv = synth.f32_to_bf16(rng.standard_normal((rows, inp.n_kv_heads, inp.head_dim), dtype=np.float32))
        self.q, self.tk, self.tv = to_device(q, dev), to_device(tk, dev), to_device(tv, dev)
        self.out = torch.empty(q.shape, dtype=torch.float32, device=dev)
        self.tail_base = tail_base
        self.bytes = (2 * int(sum((t + D) * (a + b) for t, a, b in zip(inp.block_tokens, inp.rank_k, inp.rank_v)))
                      + 4 * rows * D + 2 * q.size)
        self.flops = (sum(2 * n_tok * inp.n_q_heads * (int(a) + int(b)) * (int(t) + inp.head_dim)
                          for t, a, b in zip(inp.block_tokens, inp.rank_k, inp.rank_v))
                      + 4 * inp.n_q_heads * inp.head_dim * sum(tail_base + j + 1 for j in range(n_tok)))
        self.ctx_tokens = sum(int(inp.block_tokens.sum()) + tail_base + j + 1 for j in range(n_tok))

    def step(self, stream):
        from paper_2609_29913_amd import milo
        milo.milo_attend_prefill(self.cache, self.table, self.q, self.tk, self.tv, self.tail_base, self.scale,
                                 self.out, stream=stream)


def run_prefill(args, cfg, dev):
    """Time the causal prefill of one chunk of args.prefill tokens (see the module text)."""
    import torch
    from paper_2609_29913_amd import milo
    x = synth.gen_layer(cfg, 0)
    tail_base = int(x.tail_len.max())
    first = PrefillLayer(x, dev, args.prefill, tail_base, 0)
    copies = max(1, int(np.ceil(args.rotate_bytes / first.bytes)))
    layers = [first] + [PrefillLayer(x, dev, args.prefill, tail_base, k) for k in range(1, copies)]
    stream = torch.cuda.current_stream()
    for k in range(1, copies):  # each copy's plan, before the warm-up
        layers[k].step(stream)
    for k in range(args.warmup):
        layers[k % copies].step(stream)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(args.steps):
        layers[k % copies].step(stream)
    torch.cuda.synchronize()
    ms_per_step = (time.perf_counter() - t0) * 1e3 / args.steps
    milo.milo_timing_enable(True)
    for k in range(args.steps):
        layers[k % copies].step(stream)
    torch.cuda.synchronize()
    att_ms, merge_ms, n_calls = milo.milo_timing_read()
    milo.milo_timing_enable(False)
    att_s = att_ms / n_calls * 1e-3
    kern_bytes = first.bytes  # the attention kernel reads every factor, the tail and the queries once
    flops = first.flops
    bound = "hbm" if flops / kern_bytes < MFMA_BF16_PEAK_TFLOPS * 1e12 / (HBM_PEAK_GBS * 1e9) else "mfma"
    gbs, tfs = kern_bytes / att_s / 1e9, flops / att_s / 1e12
    result = {
        "metric": "effective context tokens/s per prefill chunk (1 GPU) + % of HBM roofline",
        "value": first.ctx_tokens / (ms_per_step * 1e-3), "unit": "tokens/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms_per_step, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic (seeded N(0,1) factors / N(0,1/r) R, queries and tail, bf16)",
        "config": {"workload": f"{cfg.name}_prefill{args.prefill}", "mode": "prefill",
                   "chunk_tokens": args.prefill, "tail_rows_before_chunk": tail_base,
                   "context_tokens": int(x.block_tokens.sum()), "blocks": x.n_blocks, "q_heads": x.n_q_heads,
                   "kv_heads": x.n_kv_heads, "head_dim": x.head_dim, "rotated_copies": copies},
        "roofline": {"bound": bound, "achieved": gbs if bound == "hbm" else tfs,
                     "peak": HBM_PEAK_GBS if bound == "hbm" else MFMA_BF16_PEAK_TFLOPS,
                     "unit": "GB/s" if bound == "hbm" else "TFLOP/s",
                     "frac": gbs / HBM_PEAK_GBS if bound == "hbm" else tfs / MFMA_BF16_PEAK_TFLOPS,
                     "traffic": None, "arithmetic_intensity_flop_per_byte": flops / kern_bytes,
                     "kernel": "attend_kernel", "kernel_avg_us": att_s * 1e6,
                     "merge_kernel_avg_us": merge_ms / n_calls * 1e3, "algorithmic_bytes_per_launch": kern_bytes,
                     "hbm_gbs": gbs, "mfma_tflops": tfs, "mfma_frac": tfs / MFMA_BF16_PEAK_TFLOPS,
                     "kernel_source_sha256_16": kernel_source_hash()},
        "cpu_baseline": None,
    }
    for layer in layers:
        milo.milo_cache_free(layer.cache)
    print(json.dumps(result), flush=True)


def run_svd(args, cfg, dev):
    """Time the encoder's per-block truncated SVD (milo_block_svd, then
    milo_block_factors at the entropy-allocated ranks) on one layer's key
    blocks of the workload's block sizes (synthetic power-law spectra)."""
    import torch
    from paper_2609_29913_amd import milo
    import oracle
    T = synth.draw_block_tokens(cfg)
    D = cfg.n_kv_heads * cfg.head_dim
    blocks = [synth.gen_kv_block(b, int(t), D, 0.9) for b, t in enumerate(T)]
    dev_blocks = [torch.from_numpy(x.view(np.int16)).to(dev) for x in blocks]
    n_sv = [min(int(t), D) for t in T]
    budget = sum(n_sv) // 2

    def encode():
        sigma, vt = milo.milo_block_svd(dev_blocks)
        ranks = milo.milo_allocate_ranks(sigma, n_sv, budget, 32, D)
        milo.milo_block_factors(dev_blocks, vt, ranks)
        return ranks

    for _ in range(args.warmup):
        encode()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        ranks = encode()
    ms = (time.perf_counter() - t0) * 1e3 / args.steps
    sweeps = milo.milo_block_svd_sweeps()
    # the SVD's own count (Gram products and the block rotations' 64 x 64 x 64
    # products, as executed), plus the factors 2 T D r
    nb = len(T)
    flops = milo.milo_block_svd_flops() + sum(2.0 * int(t) * D * int(r) for t, r in zip(T, ranks))
    tfs = flops / (ms * 1e-3) / 1e12
    cpu = None
    if not args.no_cpu_baseline:
        t1 = time.perf_counter()
        oracle.block_svd(synth.bf16_to_f64(blocks[0]))
        t_one = time.perf_counter() - t1
        cpu = {"value": 1.0 / (t_one * nb), "unit": "layers/s", "cores": 1, "kind": "oracle",
               "sample": f"one {int(T[0])} x {D} block through the fp64 one-sided Jacobi SVD ({t_one:.1f} s), "
                         f"extrapolated x{nb} blocks", "extrapolated": True}
    result = {
        "metric": "encoder layers per second (per-block truncated SVD + rank allocation + factors, 1 GPU)",
        "value": 1e3 / ms, "unit": "layers/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": ms, "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32",
        "data": "synthetic key blocks with power-law spectra (seeded), the workload's block sizes",
        "config": {"workload": f"{cfg.name}_svd", "blocks": nb, "d_model": D, "tokens": int(np.sum(T)),
                   "jacobi_sweeps_max": sweeps, "rank_budget": budget},
        "roofline": {"bound": "alu", "achieved": tfs, "peak": 157.3, "unit": "TFLOP/s", "frac": tfs / 157.3,
                     "traffic": None, "kernel": "bj_solve_kernel + bj_apply_kernel (with gram_kernel, factor_kernel)",
                     "flops_per_step": flops,
                     "note": "fp32 VALU work of the whole encode over its wall time: Gram and factor products and the "
                             "block rotations' 64^3 products as executed; the scalar rotations inside the 64 x 64 "
                             "subproblems are not counted"},
        "cpu_baseline": cpu,
    }
    print(json.dumps(result), flush=True)


def run_alloc(args, cfg, dev):
    """Time the encoder's entropy rank allocation (milo_allocate_ranks) on one
    layer's synthetic key spectra of the workload's block structure."""
    import torch
    from paper_2609_29913_amd import milo
    import oracle
    sp = synth.gen_spectra(cfg, 0)
    sig = torch.from_numpy(sp.sigma).to(dev)
    call = lambda: milo.milo_allocate_ranks(sig, sp.n_sv, sp.r_total, sp.r_min, sp.r_max)
    for _ in range(args.warmup):
        call()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        ranks = call()
    ms_per_call = (time.perf_counter() - t0) * 1e3 / args.steps
    milo.milo_timing_read_alloc()
    milo.milo_timing_enable(True)
    for _ in range(args.steps):
        call()
    milo.milo_timing_enable(False)
    chain_ms, hist_ms, n_calls = milo.milo_timing_read_alloc()
    n_values = int(sp.n_sv.sum())
    # one histogram pass must read every singular value once (the first pass
    # checks them all, the others select among the candidates of the same rows)
    pass_bytes = 4 * n_values
    hist_s = hist_ms / (4 * n_calls) * 1e-3
    chain_s = chain_ms / n_calls * 1e-3
    alloc_bytes = 4 * n_values + 4 * len(sp.n_sv)  # the whole allocation: values once, ranks out
    gbs = pass_bytes / hist_s / 1e9
    budget = 10.0 if args.cpu_budget is None else args.cpu_budget
    cpu = None
    if not args.no_cpu_baseline:
        rows = [sp.sigma[b, :n].astype(np.float64) for b, n in enumerate(sp.n_sv)]
        times, t_start = [], time.perf_counter()
        while not times or (time.perf_counter() - t_start < budget and len(times) < 20):
            t1 = time.perf_counter()
            ref = oracle.allocate_ranks(rows, sp.r_total, sp.r_min, sp.r_max)
            times.append(time.perf_counter() - t1)
        if not np.array_equal(ref, ranks):
            raise RuntimeError("allocation differs from the oracle")
        cpu = {"value": 1.0 / float(np.median(times)), "unit": "allocations/s", "cores": 1, "kind": "oracle",
               "sample": f"the same allocation (greedy over marginal gains, numpy, one thread), "
                         f"{len(times)} runs, median"}
    result = {
        "metric": "entropy rank allocations per second (one layer's blocks, 1 GPU) + % of HBM roofline",
        "value": 1e3 / ms_per_call, "unit": "allocations/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms_per_call, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "f32",
        "data": "synthetic power-law singular-value spectra with ties (seeded), the workload's block sizes",
        "config": {"workload": f"{cfg.name}_rank_allocation", "mode": "allocation", "blocks": len(sp.n_sv),
                   "singular_values": n_values, "budget": sp.r_total, "r_min": sp.r_min, "r_max": sp.r_max,
                   "ms_per_call_includes": "host checks, workspace hipMalloc/hipFree, upload, kernels, "
                                           "read-back, synchronisation"},
        "roofline": {"bound": "hbm", "achieved": gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": gbs / HBM_PEAK_GBS, "traffic": None, "kernel": "alloc_hist_kernel",
                     "kernel_avg_us": hist_s * 1e6, "algorithmic_bytes_per_launch": pass_bytes,
                     "chain_avg_us": chain_s * 1e6, "chain_algorithmic_bytes": alloc_bytes,
                     "chain_hbm_frac": alloc_bytes / chain_s / 1e9 / HBM_PEAK_GBS,
                     "kernel_source_sha256_16": kernel_source_hash(ALLOC_SOURCES)},
        "cpu_baseline": cpu,
    }
    print(json.dumps(result), flush=True)


def cpu_baseline(inp: synth.LayerInputs, n_layers: int, budget_s: float):
    """The CPU oracle (numpy, latent order, run in fp32 on fp32 copies of the
    bf16 inputs) timed on this host on the same workload.  A single-layer
    workload is timed whole; a multi-layer one on layer 0 for query 0 with all
    its heads, then scaled linearly by (n_q * H_q / H_q) columns and by the
    layers (labelled extrapolated).  Repeated until ~budget_s of CPU work."""
    import oracle
    from threadpoolctl import threadpool_info
    f32 = synth.bf16_to_f32
    args = dict(pk=[f32(x) for x in inp.pk], rk=[f32(x) for x in inp.rk], pv=[f32(x) for x in inp.pv],
                rv=[f32(x) for x in inp.rv], table=list(range(inp.n_blocks)), q=f32(inp.q),
                tail_k=f32(inp.tail_k), tail_v=f32(inp.tail_v), tail_len=inp.tail_len, scale=inp.scale)
    sampled = n_layers > 1
    if sampled:
        args["columns"] = [(0, h) for h in range(inp.n_q_heads)]
    times = []
    t_start = time.perf_counter()
    while not times or (time.perf_counter() - t_start < budget_s and len(times) < 50):
        t0 = time.perf_counter()
        oracle.attend_latent(**args)
        times.append(time.perf_counter() - t0)
    t_run = float(np.median(times))
    scale_up = inp.n_q * n_layers if sampled else 1          # columns and layers the sample stands for
    t_step = t_run * scale_up
    tokens = inp.n_q * (int(inp.block_tokens.sum()) + int(inp.tail_len.max()))
    threads = max([i.get("num_threads", 1) for i in threadpool_info() if i.get("user_api") == "blas"] or [1])
    sample = (f"layer 0, query 0 with all {inp.n_q_heads} heads (fp32 numpy oracle, latent order), "
              f"{len(times)} repetitions, median {t_run * 1e3:.1f} ms, extrapolated x{inp.n_q} queries "
              f"x{n_layers} layers" if sampled else
              f"full layer step (fp32 numpy oracle, latent order), {len(times)} repetitions, median "
              f"{t_run * 1e3:.1f} ms")
    return {"value": tokens / t_step, "unit": "tokens/s", "cores": int(threads), "host_cores": os.cpu_count(),
            "kind": "oracle", "precision": "fp32", "extrapolated": sampled, "sample": sample}


def device_env(dev, n_bytes=1 << 30, reps=5):
    """Host, software and device facts for the record, plus the bandwidth of a plain
    1 GiB device copy (bytes read + written per second: what HBM sustains here)."""
    import platform
    import socket
    import torch
    props = torch.cuda.get_device_properties(dev)
    a = torch.empty(n_bytes // 4, dtype=torch.float32, device=dev).fill_(1.0)
    b = torch.empty_like(a)
    b.copy_(a)
    st, en = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    st.record()
    for _ in range(reps):
        b.copy_(a)
    en.record()
    torch.cuda.synchronize()
    copy_gbs = 2 * n_bytes * reps / (st.elapsed_time(en) * 1e-3) / 1e9
    del a, b
    torch.cuda.empty_cache()
    return {"host": socket.gethostname(), "python": platform.python_version(), "torch": torch.__version__,
            "hip": getattr(torch.version, "hip", None), "gpu": props.name,
            "arch": getattr(props, "gcnArchName", None), "compute_units": props.multi_processor_count,
            "device_copy_gbs": copy_gbs, "gpu_clocks": gpu_clocks()}


def gpu_clocks():
    """Graphics clock levels the driver offers (sysfs pp_dpm_sclk of the first
    card that has one, MHz) and the level active when read (between runs the
    GPU idles at its lowest), or None.  Read from sysfs: no child process."""
    import glob
    for path in sorted(glob.glob("/sys/class/drm/card*/device/pp_dpm_sclk")):
        try:
            body = open(path).read()
        except OSError:
            continue
        levels = [(int(m.group(1)), "*" in m.group(0)) for m in re.finditer(r"(\d+)\s*Mhz\s*\*?", body, re.I)]
        if levels:
            return {"sclk_levels_mhz": [v for v, _ in levels], "sclk_max_mhz": max(v for v, _ in levels),
                    "sclk_active_when_read_mhz": next((v for v, cur in levels if cur), None), "source": path}
    return None


def calibrate_copy(dev, n_bytes=1 << 30, reps=5):
    """Plain device copy of known size (for scaling HBM byte counters)."""
    import torch
    a = torch.empty(n_bytes // 4, dtype=torch.float32, device=dev).fill_(1.0)
    b = torch.empty_like(a)
    for _ in range(reps):
        b.copy_(a)
    torch.cuda.synchronize()
    print(json.dumps({"calibration_copy_bytes_read": n_bytes, "bytes_written": n_bytes, "reps": reps}))


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=None,
                    help="timed steps (default 500 for a single-layer workload, else 10)")
    ap.add_argument("--warmup", type=int, default=None,
                    help="untimed steps first (default 200 for a single-layer workload, else 2); the "
                         "kernels reach their steady-state speed after ~100 back-to-back steps")
    ap.add_argument("--config", default="q32b_64l", choices=sorted(synth.CONFIGS),
                    help="workload (default: the largest that fits one GPU, the 32B-shaped 64-layer step)")
    ap.add_argument("--int8", action="store_true",
                    help="store P^K and P^V as INT8 codes with per-token scales (MILO_P_INT8)")
    ap.add_argument("--path", choices=sorted(PATHS), default="latent",
                    help="how blocks are attended: latent (rank space), reconstruct (full-rank K/V rebuilt "
                         "per step, Sec. 4.5) or auto (per block, by the library's cost model)")
    ap.add_argument("--rope", type=float, default=0.0, metavar="THETA",
                    help="keys stored before the rotary embedding (base THETA, e.g. 1e6): every block is "
                         "reconstructed and its keys rotated to their positions (milo_cache_set_rope)")
    ap.add_argument("--grow-tails", action="store_true",
                    help="decode loop: every request's tail grows by one token per step (warm-up and timed "
                         "steps), ending at the workload's tail length")
    ap.add_argument("--rotate-bytes", type=float, default=512e6,
                    help="minimum bytes of distinct layer copies rotated over (defeats the Infinity Cache)")
    ap.add_argument("--cpu-budget", type=float, default=10.0, help="seconds of oracle work for cpu_baseline")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--calibrate-copy", action="store_true", help="only run a 1 GiB device copy (counter scaling)")
    ap.add_argument("--prefill", type=int, default=0, metavar="N",
                    help="time the causal prefill of an N-token chunk of one request instead (first layer)")
    ap.add_argument("--svd", action="store_true",
                    help="time the encoder's per-block truncated SVD (Gram matrix, Jacobi, factors) on one layer's "
                         "key blocks of the workload instead (default workload then: the 7B-shaped layer)")
    ap.add_argument("--alloc", action="store_true",
                    help="time the encoder's entropy rank allocation on the workload's block structure instead")
    args = ap.parse_args()

    if args.gpus != 1:
        print(f"bench.py: this decode-attention path runs on one GPU; --gpus {args.gpus} is not supported "
              "(sharding by blocks across GPUs is not built).", file=sys.stderr)
        sys.exit(2)

    import torch
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    if args.calibrate_copy:
        calibrate_copy(dev)
        return
    from paper_2609_29913_amd import milo
    milo.lib()

    if args.svd and args.config == ap.get_default("config"):
        args.config = "q7b_1l"
    cfg = synth.CONFIGS[args.config]
    if args.steps is None:
        args.steps = 3 if args.svd else 200 if args.alloc else 500 if cfg.n_layers == 1 else 10
    if args.warmup is None:
        args.warmup = 1 if args.svd else 20 if args.alloc else 200 if cfg.n_layers == 1 else 2
    if args.svd:
        run_svd(args, cfg, dev)
        return
    if args.prefill > 0:
        run_prefill(args, cfg, dev)
        return
    if args.alloc:
        run_alloc(args, cfg, dev)
        return
    # layers are generated one at a time and only their device state is kept
    # (a 64-layer workload's host factors would not fit next to each other)
    grow_from = 0
    if args.grow_tails:
        grow_from = max(1, cfg.tail - (args.warmup + args.steps) + 1)
    x0 = None
    per_step = flops_step = recon_flops_step = out_bytes = 0
    mean_ranks = []
    groups = [[]]
    t_gen = time.perf_counter()
    t_make = 0.0
    for l in range(cfg.n_layers):
        x = synth.gen_layer(cfg, l)
        per_step += synth.algorithmic_bytes(x, p_int8=args.int8)
        flops_step += synth.latent_flops(x)
        recon_flops_step += synth.recon_flops(x)
        out_bytes += 4 * x.n_q * x.n_q_heads * x.head_dim
        mean_ranks.append(float(x.rank_k.mean()))
        t1 = time.perf_counter()
        groups[0].append(Layer(x, dev, args.int8, args.path, args.rope))
        t_make += time.perf_counter() - t1
        if cfg.n_layers > 1:
            print(f"bench: layer {l + 1}/{cfg.n_layers} ready ({time.perf_counter() - t_gen:.0f} s, "
                  f"{t_make:.1f} s of it in milo_cache_create)", file=sys.stderr, flush=True)
        if l == 0:
            x0 = x
    copies = max(1, int(np.ceil(args.rotate_bytes / per_step)))
    for _ in range(1, copies):
        groups.append([Layer(synth.gen_layer(cfg, l), dev, args.int8, args.path, args.rope)
                       for l in range(cfg.n_layers)])
    stream = torch.cuda.current_stream()
    if args.grow_tails:
        for grp in groups:
            for layer in grp:
                layer.tail_len = np.full_like(layer.tail_len, grow_from - 1)
    torch.cuda.synchronize()
    host_s = [0.0]

    def run_step(k, grow=0):
        for layer in groups[k % copies]:
            h0 = time.perf_counter()
            layer.step(stream, grow)
            host_s[0] += time.perf_counter() - h0

    grow = 1 if args.grow_tails else 0
    # every rotated copy is a cache of its own: build each one's plan once
    # before the warm-up (with fewer warm-up steps than copies, the first call
    # on a copy would otherwise fall into the timed region)
    for k in range(1, copies):
        run_step(k, 0)
    for k in range(args.warmup):
        run_step(k, grow)
    torch.cuda.synchronize()

    # timed region: exactly `steps` decode steps, host wall clock between synchronisations
    builds0 = sum(milo.milo_cache_plan_builds(layer.cache) for grp in groups for layer in grp)
    host_s[0] = 0.0
    tail_sum = 0
    t0 = time.perf_counter()
    for k in range(args.steps):
        run_step(k, grow)
        tail_sum += int(groups[k % copies][0].tail_len.max())
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    ms_per_step = elapsed * 1e3 / args.steps
    host_us_per_call = host_s[0] * 1e6 / (args.steps * cfg.n_layers)
    plan_builds = sum(milo.milo_cache_plan_builds(layer.cache) for grp in groups for layer in grp) - builds0
    mean_tail = tail_sum / args.steps

    # host cost of a call with the device idle: one step enqueued after a
    # synchronisation, a few times (the timed loop above runs ahead of the GPU
    # until launches wait for queue space, so it cannot show this)
    enq = []
    for k in range(min(args.steps, 5)):
        torch.cuda.synchronize()
        h0 = time.perf_counter()
        run_step(k)
        enq.append(time.perf_counter() - h0)
    torch.cuda.synchronize()
    host_idle_us_per_call = float(np.median(enq)) * 1e6 / cfg.n_layers

    # second pass with HIP events around the attention kernel on the launch stream
    milo.milo_timing_enable(True)
    for k in range(args.steps):
        run_step(k)
    torch.cuda.synchronize()
    att_ms, merge_ms, n_calls = milo.milo_timing_read()
    recon_ms, _ = milo.milo_timing_read_recon()
    milo.milo_timing_enable(False)
    recon_blocks = sum(milo.milo_cache_recon_blocks(layer.cache) for layer in groups[0])
    att_avg_s = att_ms / n_calls * 1e-3
    merge_avg_s = merge_ms / n_calls * 1e-3

    # third pass: each step between HIP events on the launch stream (distribution)
    import torch
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    evs[0].record(stream)
    for k in range(args.steps):
        run_step(k)
        evs[k + 1].record(stream)
    torch.cuda.synchronize()
    step_us = np.array([evs[k].elapsed_time(evs[k + 1]) * 1e3 for k in range(args.steps)])

    # the attention kernel reads every factor once, the tails and the queries
    kern_bytes = (per_step - out_bytes) / cfg.n_layers
    flops = flops_step / cfg.n_layers
    achieved = kern_bytes / att_avg_s / 1e9
    mfma_tflops = flops / att_avg_s / 1e12
    # the bound is the roof the kernel's arithmetic intensity meets first
    bound = "hbm" if flops / kern_bytes < MFMA_BF16_PEAK_TFLOPS * 1e12 / (HBM_PEAK_GBS * 1e9) else "mfma"
    traffic, mfma_busy = counter_values(workload_name(cfg, args))
    t_roof = max(kern_bytes / (HBM_PEAK_GBS * 1e9), flops / (MFMA_BF16_PEAK_TFLOPS * 1e12))

    ctx_tokens = int(x0.block_tokens.sum()) + (mean_tail if args.grow_tails else int(x0.tail_len.max()))
    value = x0.n_q * ctx_tokens / (ms_per_step * 1e-3)
    result = {
        "metric": METRIC,
        "value": value,
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded N(0,1) factors / N(0,1/r) R, bf16)",
        "config": {
            "workload": workload_name(cfg, args),
            "p_factors": "int8 codes + per-token fp32 scales" if args.int8 else "bf16",
            "description": cfg.description,
            "layers": cfg.n_layers,
            "decode_batch": x0.n_q,
            "context_tokens": int(x0.block_tokens.sum()),
            "tail_tokens": int(x0.tail_len.max()),
            "blocks": x0.n_blocks,
            "q_heads": x0.n_q_heads,
            "kv_heads": x0.n_kv_heads,
            "head_dim": x0.head_dim,
            "mean_rank": float(np.mean(mean_ranks)),
            "accumulation": "fp32",
            "rotated_copies": copies,
            "step_bytes_algorithmic": per_step,
            "hbm_frac_of_step": per_step / (ms_per_step * 1e-3) / (HBM_PEAK_GBS * 1e9),
        },
        "step_us": {"median": float(np.median(step_us)), "min": float(step_us.min()),
                    "p90": float(np.percentile(step_us, 90)), "timing": "HIP events between steps"},
        "host": {"us_per_call": host_idle_us_per_call, "us_per_call_in_timed_loop": host_us_per_call,
                 "plan_builds_in_timed_steps": plan_builds,
                 "tails": (f"growing one token per step, {grow_from}..{cfg.tail} (mean {mean_tail:.0f} in the "
                           f"timed steps)") if args.grow_tails else "fixed",
                 "timing": "host wall time inside milo_attend_decode calls (binding, checks, launches): "
                           "us_per_call with the device idle (median over 5 steps enqueued after a "
                           "synchronisation); in the timed loop it also holds waits for launch-queue space"},
        "roofline": {
            "bound": bound,
            "achieved": achieved if bound == "hbm" else mfma_tflops,
            "peak": HBM_PEAK_GBS if bound == "hbm" else MFMA_BF16_PEAK_TFLOPS,
            "unit": "GB/s" if bound == "hbm" else "TFLOP/s",
            "frac": achieved / HBM_PEAK_GBS if bound == "hbm" else mfma_tflops / MFMA_BF16_PEAK_TFLOPS,
            "traffic": traffic,
            "arithmetic_intensity_flop_per_byte": flops / kern_bytes,
            "kernel": "attend_kernel",
            "kernel_avg_us": att_avg_s * 1e6,
            "merge_kernel_avg_us": merge_avg_s * 1e6,
            "algorithmic_bytes_per_launch": kern_bytes,
            "hbm_gbs": achieved,
            "mfma_tflops": mfma_tflops,
            "mfma_frac": mfma_tflops / MFMA_BF16_PEAK_TFLOPS,
            "hbm_frac": achieved / HBM_PEAK_GBS,
            "mfma_busy_counter": mfma_busy,
            "counters": (os.path.relpath(counter_summary(workload_name(cfg, args)), ROOT)
                         if traffic is not None else None),
            "attainable_frac": t_roof / att_avg_s,
            "kernel_source_sha256_16": kernel_source_hash(),
        },
        "cpu_baseline": None,
    }
    if args.path != "latent" or args.rope > 0:
        # the route's own work: rebuilt blocks do 2 T D (rk + rv) flops of
        # reconstruction and 4 N T d of dense attention instead of the latent
        # 2 N (rk + rv)(T + d); the roofline above prices the latent work
        recon_avg_s = recon_ms / n_calls * 1e-3
        result["roofline"]["note"] = ("latent accounting: the latent route's bytes and flops over the attention "
                                      "kernel alone; with reconstructed blocks that is not the work done (the "
                                      "route object gives the reconstruction time and, for every block rebuilt, "
                                      "the route's own flops)")
        result["route"] = {
            "path": "reconstruct, pre-RoPE keys rotated" if args.rope > 0 else args.path,
            "reconstructed_blocks_per_step": recon_blocks,
            "blocks_per_step": x0.n_blocks * cfg.n_layers,
            "recon_kernel_avg_us": recon_avg_s * 1e6,
            "attend_plus_recon_us": (att_avg_s + recon_avg_s) * 1e6,
        }
        if args.path == "reconstruct" or args.rope > 0:
            rflops = recon_flops_step / cfg.n_layers
            result["route"]["route_flops_per_layer"] = rflops
            result["route"]["route_tflops"] = rflops / (att_avg_s + recon_avg_s) / 1e12
            result["route"]["route_mfma_frac"] = rflops / (att_avg_s + recon_avg_s) / 1e12 / MFMA_BF16_PEAK_TFLOPS
    for grp in groups:
        for layer in grp:
            milo.milo_cache_free(layer.cache)
    result["env"] = device_env(dev)
    if not args.no_cpu_baseline and args.rope == 0:  # the oracle baseline times the unrotated latent order
        result["cpu_baseline"] = cpu_baseline(x0, cfg.n_layers, args.cpu_budget)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
