#!/usr/bin/env python3
"""Benchmark of paged grouped-query decode attention on one MI355X.

One step is one pass of the whole hot path over one batch: plan the split of
the batch's KV pages across CUs (host), upload the work list, run the split-KV
partial kernel and the log-sum-exp merge. Inputs are generated on the GPU
before timing and stay resident in HBM.

Default workload: 256 trajectories with lognormal(median 2048, sigma 1)
lengths clipped to [16, 32768], 28 query / 4 KV heads, head_dim 128, bf16 KV
(a 7B-class rollout step before repack). Prints ONE JSON line: the
headline workload's figures, then `per_config`, one row per workload (all
seven by default) with its step, kernel and merge times, fractions of HBM
peak, committed HBM traffic ratio and its errors against the fp64 oracle
over every trajectory.

    python bench.py [--steps K] [--warmup W] [--workload NAME|N]
"""
from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import platform
import random
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "decode-attn KV TB/s (fraction of HBM peak) + tokens/s at long-tail batch"
HBM_PEAK_GBPS = 8000.0          # MI355X HBM3E, published
PARITY_TOL = 1e-3               # max-abs error of fp32 out and lse vs the oracle
DEFAULT_WORKLOAD = "7b_pre_repack"
PARTIAL_KERNEL = "decode_items"
PROFILE_DIR = os.path.join(ROOT, "profiles")
# The attention kernels and the planner that shapes and orders their work:
# the committed counters and kernel statistics hold for these sources.
KERNEL_SOURCES = tuple(os.path.join(ROOT, "paper_2510_12633_amd", "csrc", f)
                       for f in ("decode_attn.hip", "plan.cpp"))


def parse_args(argv=None):
    p = argparse.ArgumentParser(description=__doc__,
                                formatter_class=argparse.RawDescriptionHelpFormatter)
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=100)
    p.add_argument("--warmup", type=int, default=20)
    p.add_argument("--workload", default=DEFAULT_WORKLOAD,
                   help="workload name or 1-based index")
    p.add_argument("--seed", type=int, default=None)
    p.add_argument("--waves-per-item", type=int, default=0)
    p.add_argument("--pages-per-item", type=int, default=0)
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--cpu-budget-s", type=float, default=15.0,
                   help="target seconds of oracle work for the CPU baseline")
    p.add_argument("--no-calibrate", action="store_true",
                   help="skip the HBM read/copy calibration kernels")
    p.add_argument("--cascade", choices=("auto", "off"), default="auto",
                   help="decode shared prompt prefixes once per group when "
                        "the workload has them (auto) or not at all (off)")
    p.add_argument("--no-append", action="store_true",
                   help="skip the KV-append timing")
    p.add_argument("--latency-curve", action="store_true",
                   help="also time full Qwen2.5-shaped decode steps over "
                        "batch sizes (the latency-versus-batch curve)")
    p.add_argument("--curve-model", choices=sorted(CURVE_MODELS),
                   default="qwen7b", help="decoder shape for --latency-curve")
    p.add_argument("--no-projections", action="store_true",
                   help="skip the skinny projection kernel timing")
    p.add_argument("--curve-batches", default="",
                   help="comma-separated batch sizes for --latency-curve")
    p.add_argument("--curve-contexts", default="",
                   help="comma-separated cached-token counts for --latency-curve")
    p.add_argument("--no-repack", action="store_true",
                   help="skip the repack planner and page-migration timing")
    p.add_argument("--fixed-plan", action="store_true",
                   help="plan once outside the timed loop (kernel-only steps)")
    p.add_argument("--no-per-config", action="store_true",
                   help="measure the named workload only, not every one")
    p.add_argument("--no-parity", action="store_true",
                   help="skip the oracle check of every trajectory")
    return p.parse_args(argv)


def source_digest() -> str:
    h = hashlib.sha256()
    for path in KERNEL_SOURCES:
        with open(path, "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def read_traffic(workload: str):
    """HBM bytes per partial-kernel launch from the committed rocprofv3
    --pmc summary, if it was taken on the current kernel source."""
    path = os.path.join(PROFILE_DIR, f"{PARTIAL_KERNEL}_{workload}_traffic.txt")
    if not os.path.exists(path):
        return None, None
    vals = {}
    with open(path) as f:
        for line in f:
            if ":" in line and not line.startswith("#"):
                k, v = line.split(":", 1)
                vals[k.strip()] = v.strip()
    if vals.get("kernel_source_sha256_16") != source_digest():
        return None, "stale"
    try:
        return float(vals["hbm_bytes_per_launch"]), path
    except (KeyError, ValueError):
        return None, None


class Rotation:
    """Copies of the KV pools so that inputs under ~2 GB are not served from
    the 256 MB Infinity Cache on back-to-back steps."""

    def __init__(self, wl, min_bytes=2 << 30):
        import torch
        pool = wl.k_pages.numel() * wl.k_pages.element_size() * 2
        n = max(1, math.ceil(min_bytes / max(pool, 1)))
        n = min(n, 64)
        self.k = [wl.k_pages] + [wl.k_pages.clone() for _ in range(n - 1)]
        self.v = [wl.v_pages] + [wl.v_pages.clone() for _ in range(n - 1)]
        self.n = n
        torch.cuda.synchronize()

    def get(self, i):
        j = i % self.n
        return self.k[j], self.v[j]


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.machine()


def cpu_baseline(wl, budget_s: float):
    """The fp64 oracle on the host over a bounded sample of the workload."""
    import numpy as np
    from threadpoolctl import threadpool_limits

    from oracle import decode_attention_from_host
    from workloads import host_arrays

    cores = len(os.sched_getaffinity(0))
    rng = random.Random(0)
    order = list(range(wl.batch))
    rng.shuffle(order)
    c = wl.cfg
    per_tok = c.num_kv_heads * c.head_dim * 2 * c.kv_elem_bytes
    with threadpool_limits(1):
        # calibrate on a few trajectories, then size the sample to the budget
        probe = order[:min(4, len(order))]
        t0 = time.perf_counter()
        decode_attention_from_host(host_arrays(wl, probe), workers=cores)
        dt = max(time.perf_counter() - t0, 1e-3)
        rate = max(int(wl.seq_lens[probe].sum()), 1) / dt       # tokens/s
        want = rate * budget_s
        sample, tot = [], 0
        for b in order:
            if tot >= want and sample:
                break
            sample.append(b)
            tot += int(wl.seq_lens[b])
        arrays = host_arrays(wl, sorted(sample))
        # repeat the pass until about budget_s of CPU time (threads x wall)
        # has been spent, at most 5 passes; report the median pass
        times = []
        while True:
            t0 = time.perf_counter()
            decode_attention_from_host(arrays, workers=cores)
            times.append(time.perf_counter() - t0)
            if len(times) >= 5 or sum(times) * cores >= budget_s:
                break
        dt = sorted(times)[len(times) // 2]
    toks = int(wl.seq_lens[sample].sum())
    return {
        "value": toks * per_tok / dt / 1e12,
        "unit": "TB/s",
        "cores": cores,
        "kind": "oracle",
        "sample": f"{len(sample)} of {wl.batch} trajectories ({toks} tokens, "
                  f"{toks * per_tok / 1e9:.3f} GB of KV), fp64 numpy, "
                  f"{cores} threads over trajectories, BLAS 1 thread each; "
                  f"median of {len(times)} passes",
        "seconds": dt,
        "tokens_per_s": len(sample) / dt,
        "cpu": cpu_model(),
    }


def calibrate(torch, N, nbytes=4 << 30, iters=10):
    """Achievable HBM bandwidth (GB/s) on this device: a sequential read, a
    copy (bytes read + written), and gathers of random 4 KiB tiles (the
    size of one bf16 (page, kv-head) KV tile at head_dim 128) and of random
    64-byte tiles through an index list, each tile of the buffer once in a
    random order (tile bytes only; the index list adds 4 bytes per tile)."""
    buf = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    buf.fill_(1)
    sink = torch.empty(N.laminar_hbm_read_sink_floats(), dtype=torch.float32,
                       device="cuda")
    s = torch.cuda.current_stream()
    h = s.cuda_stream

    def timed(fn, moved):
        for _ in range(2):
            fn()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(s)
        for _ in range(iters):
            fn()
        e1.record(s)
        torch.cuda.synchronize()
        return moved * iters / (e0.elapsed_time(e1) / 1e3) / 1e9

    res = {"read": timed(lambda: N.laminar_hbm_read(buf, nbytes, sink, h),
                         nbytes)}
    half = nbytes // 2
    dst, src = buf[:half], buf[half:]
    res["copy"] = timed(lambda: N.laminar_hbm_copy(dst, src, half, h), 2 * half)
    gen = torch.Generator(device="cuda").manual_seed(7)
    for tile, span in ((4096, nbytes), (64, 1 << 30)):
        n = span // tile
        idx = torch.randperm(n, generator=gen, device="cuda").to(torch.int32)
        gsink = torch.empty(N.laminar_hbm_gather_sink_words(n, tile),
                            dtype=torch.int32, device="cuda")
        key = "gather_4KiB" if tile == 4096 else "gather_64B"
        res[key] = timed(lambda: N.laminar_hbm_gather(buf, nbytes, tile, idx,
                                                      n, gsink, h), span)
        del idx, gsink
    del buf
    torch.cuda.empty_cache()
    return res


def graph_launch_floor(torch, chain=100, reps=20):
    """What one kernel costs in a captured graph when it does almost
    nothing: a chain of `chain` in-place adds on 4 KiB and on 1 MiB,
    captured once and replayed `reps` times; microseconds per kernel."""
    side = torch.cuda.Stream()
    res = {}
    for label, nbytes in (("4KiB", 4096), ("1MiB", 1 << 20)):
        x = torch.zeros(nbytes // 4, device="cuda")
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            for _ in range(3):
                x.add_(1.0)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=side):
            for _ in range(chain):
                x.add_(1.0)
        torch.cuda.synchronize()
        for _ in range(3):
            g.replay()
        torch.cuda.synchronize()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            g.replay()
        e1.record()
        torch.cuda.synchronize()
        res[label] = round(1e3 * e0.elapsed_time(e1) / (reps * chain), 2)
        del g, x
    return res


def measure_append(torch, wl, steps=24):
    """Time the KV append (one launch per decode step) on this workload's
    pools, copied and grown by ``steps`` tokens per trajectory. Returns None
    for workloads with shared prefix pages (a shared last page would need a
    copy before it is written)."""
    from paper_2510_12633_amd.api import kv_append
    from workloads import make_decode_run
    if wl.cfg.prefix_group:
        return None
    run = make_decode_run(wl, steps=steps, seed=11, mix="normal")
    dev = run.k_pages.device
    bt = torch.as_tensor(run.block_table, device=dev)
    lens = [torch.as_tensor(run.lens_after(i), device=dev) for i in range(steps)]
    stream = torch.cuda.current_stream()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    warm = 4

    def append(i):
        kv_append(run.k_new[i], run.v_new[i], bt, lens[i], run.k_pages,
                  run.v_pages, run.k_scale, run.v_scale,
                  kv_dtype=wl.cfg.kv_dtype, stream=stream)
    for i in range(warm):
        append(i)
    # back-to-back launches between two events (one decode step each)
    e0.record(stream)
    for i in range(warm, steps):
        append(i)
    e1.record(stream)
    torch.cuda.synchronize()
    times = [e0.elapsed_time(e1) / (steps - warm)] * (steps - warm)
    us = 1e3 * sum(times) / len(times)
    c = wl.cfg
    units = wl.batch * c.num_kv_heads
    e = 1 if c.kv_dtype == "fp8_e4m3fn" else 2
    nbytes = (units * c.head_dim * 2 * 2            # new K and V, bf16
              + units * c.head_dim * e * 2          # their slots in the pages
              + wl.batch * 8                        # table entry + length
              + (units * 2 * 4 * 2 if e == 1 else 0))   # scales read + written
    del run
    return {"kernel": "kv_append_kernel", "us_per_call": round(us, 3),
            "algorithmic_bytes_per_call": nbytes,
            "GBps": round(nbytes / (us * 1e-6) / 1e9, 1),
            "bound": "launch/latency (a few hundred bytes per trajectory)",
            "timed_calls": len(times)}


def measure_repack(torch, N, wl, n_rollouts=256, reps=50):
    """Repack legs: the consolidation planner's host time for n_rollouts
    rollout states, and the page migration kernel moving this workload's
    whole pool (K, V and any scales) into a second pool in a random page
    order."""
    import ctypes
    import numpy as np
    rng = np.random.default_rng(5)
    used = rng.integers(100, 60000, n_rollouts)
    states = (N.LaminarRolloutState * n_rollouts)()
    for i in range(n_rollouts):
        states[i].kv_used = int(used[i])
        states[i].kv_prev = int(used[i] + rng.integers(-500, 3000))
        states[i].num_reqs = int(rng.integers(1, 300))
    src = (ctypes.c_int32 * n_rollouts)()
    dst = (ctypes.c_int32 * n_rollouts)()
    k = ctypes.c_int32()
    lib = N.lib()
    best = float("inf")
    for _ in range(reps):
        t0 = time.perf_counter_ns()
        st = lib.laminar_repack_plan(states, n_rollouts, 65536, 256, src, dst,
                                     ctypes.byref(k))
        best = min(best, time.perf_counter_ns() - t0)
        assert st == N.LAMINAR_OK

    pools = [t for t in (wl.k_pages, wl.v_pages, wl.k_scale, wl.v_scale)
             if t is not None]
    n = pools[0].shape[0]
    dev = pools[0].device
    perm = torch.randperm(n, generator=torch.Generator().manual_seed(1))
    pairs = torch.stack([torch.arange(n), perm], dim=1).to(torch.int32).to(dev)
    dsts = [torch.empty_like(t) for t in pools]
    stream = torch.cuda.current_stream()
    h = stream.cuda_stream

    def run():
        for s_, d_ in zip(pools, dsts):
            N.laminar_migrate_pages(s_, n, d_, n, s_[0].numel() * s_.element_size(),
                                    pairs, n, h)

    run()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    iters = 5
    e0.record(stream)
    for _ in range(iters):
        run()
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / iters
    nbytes = 2 * sum(t.numel() * t.element_size() for t in pools)   # read + write
    for s_, d_ in zip(pools, dsts):
        # bytes, not values: the pools hold NaN poison in unused slots
        assert torch.equal(d_.view(torch.uint8)[pairs[:, 1].long()],
                           s_.view(torch.uint8))
    del dsts
    torch.cuda.empty_cache()
    return {"plan_us": round(best / 1e3, 2), "rollouts": n_rollouts,
            "pairs_planned": k.value,
            "migrate": {"kernel": "migrate_kernel16", "pages": n,
                        "bytes_read_plus_written": nbytes,
                        "ms": round(ms, 4),
                        "GBps": round(nbytes / (ms / 1e3) / 1e9, 1),
                        "frac_of_hbm_peak": round(nbytes / (ms / 1e3) / 1e9
                                                  / HBM_PEAK_GBPS, 4)}}


QWEN7B_PROJECTIONS = {"qkv": (4608, 3584), "o": (3584, 3584),
                      "gate_up": (37888, 3584), "down": (3584, 18944),
                      "lm_head": (152064, 3584)}


def measure_projections(torch, N, batches=(1, 16, 64, 128), reps=20):
    """The skinny projection kernel on Qwen2.5-7B's projection shapes (w
    [N, K] bf16, packed once), HIP-event time per call and weight bytes /
    time, next to the library GEMM (torch.matmul) on the same operands.
    Calls cycle over enough copies of each weight (at least 512 MB) that
    the 256 MB Infinity Cache cannot serve them, as in a decode step that
    runs every layer once."""
    from paper_2510_12633_amd.api import SkinnyLinear
    gen = torch.Generator(device="cuda").manual_seed(9)
    stream = torch.cuda.current_stream()
    rows = []
    for name, (n, k) in QWEN7B_PROJECTIONS.items():
        wbytes = 2 * n * k
        copies = max(1, -(-(512 << 20) // wbytes))
        lins, wts = [], []
        for _ in range(copies):
            w = torch.randn((n, k), generator=gen, device="cuda").to(torch.bfloat16)
            wts.append(w.t().contiguous())         # [K, N] for x @ wt
            lins.append(SkinnyLinear(w))
            del w
        calls = max(reps, 2 * copies)
        for m in batches:
            x = torch.randn((m, k), generator=gen, device="cuda").to(torch.bfloat16)
            out = torch.empty((m, n), device="cuda")
            for fn_name, fn in (("laminar_linear", lambda i: lins[i % copies](x, out=out)),
                                ("library_gemm", lambda i: x @ wts[i % copies])):
                for i in range(copies):
                    fn(i)
                e0 = torch.cuda.Event(enable_timing=True)
                e1 = torch.cuda.Event(enable_timing=True)
                e0.record(stream)
                for i in range(calls):
                    fn(i)
                e1.record(stream)
                torch.cuda.synchronize()
                us = 1e3 * e0.elapsed_time(e1) / calls
                rows.append({"proj": name, "n": n, "k": k, "m": m,
                             "impl": fn_name, "us": round(us, 2),
                             "weight_copies": copies,
                             "weight_GBps": round(wbytes / (us * 1e-6) / 1e9, 1),
                             "frac_hbm_peak": round(wbytes / (us * 1e-6) / 1e9
                                                    / HBM_PEAK_GBPS, 4)})
        del lins, wts
        torch.cuda.empty_cache()
    return rows


CURVE_MODELS = {
    # layers, hidden, q heads, kv heads, head dim, intermediate, vocab
    "qwen7b": ("Qwen2.5-7B", (28, 3584, 28, 4, 128, 18944, 152064)),
    "qwen32b": ("Qwen2.5-32B", (64, 5120, 40, 8, 128, 27648, 152064)),
}


def latency_curve(torch, N, batches=(1, 2, 4, 8, 16, 32, 64, 128, 256, 384,
                                     512, 768, 1024),
                  contexts=(16, 2048), reps=5, model="qwen7b"):
    """One decode step of a Qwen2.5-7B- or 32B-shaped decoder (28 or 64
    layers, all on this one GPU, random bf16 weights; per layer this
    library's RMS pre-norms, the QKV, O, gate+up and down projections (the
    O and down ones adding the residual stream), its KV append, paged
    attention and SwiGLU; then the LM head) captured in a HIP graph and
    timed at each batch size. Each projection kind runs the faster of this library's
    skinny kernel (batches up to 128) and the library GEMM, timed first at
    that batch; next to the roofline model's step
    time and batch bound. Every replay is checked bit for bit against the
    eager step. Every trajectory holds `context` cached tokens; one KV pool
    serves all layers (the bytes read per layer are those of a real step).
    Rotary embedding and biases are left out."""
    import numpy as np
    from paper_2510_12633_amd.api import (PagedDecodeAttention, kv_append,
                                          kv_append_desc)
    model_name, (L, h, hq, hkv, d, inter, vocab) = CURVE_MODELS[model]
    shape = N.LaminarModelShape(layers=L, hidden=h, q_heads=hq, kv_heads=hkv,
                                head_dim=d, intermediate=inter, vocab=vocab,
                                weight_bytes=2, act_bytes=2, kv_bytes=2)
    peak_f, peak_bw = 2_500_000_000_000_000, 8_000_000_000_000
    bound = N.laminar_roofline_batch_bound(shape, peak_f, peak_bw)
    gen = torch.Generator(device="cuda").manual_seed(3)
    # Let PyTorch's TunableOp pick the library GEMM's kernel per shape (it
    # times the candidate hipBLASLt / rocBLAS solutions on first use, here
    # during the untimed warm-up calls): the comparison is against the
    # library at its best, and the large batches run faster with it.
    tunable = getattr(torch.cuda, "tunable", None)
    if tunable is not None:
        tunable.enable(True)
        tunable.tuning_enable(True)
        tunable.set_max_tuning_duration(30)
        tunable.set_filename(os.path.join(
            os.environ.get("TMPDIR", "/tmp"), "laminar_tunableop.csv"))
    bf = torch.bfloat16

    from paper_2510_12633_amd.api import SkinnyLinear, rmsnorm, silu_mul

    class Proj:
        """One projection's weight in two layouts: packed by this library's
        skinny kernel, and [K, N] for the library GEMM (x @ w). `mode` says
        which runs: "library", "skinny" (after a separate cast or SwiGLU
        launch when the input needs one) or "fused" (the skinny kernel
        makes its operand from the fp32 or gate-and-up input on load)."""

        def __init__(self, k, n):
            nk = (torch.randn((n, k), generator=gen, device="cuda",
                              dtype=bf) * (1.0 / k ** 0.5))
            self.k = k
            self.kn = nk.t().contiguous()
            self.skinny = SkinnyLinear(nk)
            del nk
            self.mode = "library"

        def __call__(self, x, residual=None, swiglu=False, norm=None,
                     operand=None, next_norm=None, swiglu_out=False,
                     append=None):
            """bf16(x w^T), plus residual when given (in place into it on
            the skinny path). fp32 x is rounded to bf16; with swiglu, x
            [M, 2K] is SwiGLU's gate and up; with norm (a [K] weight), the
            operand is the RMS norm of x, unless `operand` hands it over
            already made (by the producer's reduction). With next_norm (a
            [N] weight) it returns (y, rmsnorm(y)) and with swiglu_out (y,
            SwiGLU of y's halves); the skinny kernel makes the second in its
            reduction launch where it has one, the other ways return None
            for it. With append (the arguments of
            SkinnyLinear.bf16_kv_append after x) the skinny path also makes
            the step's KV append and sets self.appended."""
            pair = next_norm is not None or swiglu_out
            mode = self.mode
            self.appended = False
            if operand is not None:
                x, swiglu, norm = operand, False, None
                mode = "skinny" if mode == "fused" else mode
            if mode == "fused":           # the operand made on load
                if next_norm is not None:
                    return self.skinny.bf16_norm(x, next_norm, out=residual,
                                                 residual=residual,
                                                 swiglu=swiglu)
                y = self.skinny.bf16(x, out=residual, residual=residual,
                                     swiglu=swiglu, norm_weight=norm)
                return (y, None) if pair else y
            if swiglu:
                x = silu_mul(x)
            elif norm is not None:
                x = rmsnorm(x, norm)
            elif x.dtype != bf:
                x = x.to(bf)
            if mode == "skinny":
                if append is not None:
                    self.appended = True
                    return self.skinny.bf16_kv_append(x, *append)
                if next_norm is not None:
                    return self.skinny.bf16_norm(x, next_norm, out=residual,
                                                 residual=residual)
                if swiglu_out:
                    return self.skinny.bf16_swiglu(x)
                return self.skinny.bf16(x, out=residual, residual=residual)
            y = x @ self.kn if residual is None else torch.addmm(residual, x, self.kn)
            return (y, None) if pair else y

    layers = [(Proj(h, (hq + 2 * hkv) * d), Proj(hq * d, h),
               Proj(h, 2 * inter), Proj(inter, h)) for _ in range(L)]
    lm_head = Proj(h, vocab)
    # RMS norm weights: before attention and before the MLP of each layer,
    # and the final one
    norms = (1 + 0.1 * torch.randn((2 * L + 1, h), generator=gen,
                                   device="cuda")).to(bf)

    def choose(m):
        """Per projection kind, the fastest way to run it at this batch:
        the library GEMM, the skinny kernel, and for O and down also the
        skinny kernel with its input made on load. Each is timed over every
        layer's weights in turn (as in a step, so the 256 MB Infinity Cache
        does not hold them), captured in a HIP graph as the step is (timed
        eagerly, the host's launches counted: the fused down projection,
        one launch, won at batch 64 while its GPU time was 10 us longer
        than SwiGLU and the bf16 call), the best of three alternating
        passes, so that one slow pass (a clock change) cannot decide."""
        picks = {}
        for i, kind in enumerate(("qkv", "o", "gate_up", "down", "lm_head")):
            projs = ([lm_head] * 4 if kind == "lm_head" else
                     [layer[i] for layer in layers])
            # the operand as the step hands it over: the residual stream
            # and a norm weight to QKV, gate+up and the LM head, the
            # attention's fp32 output to O, gate and up to down
            normed = kind in ("qkv", "gate_up", "lm_head")
            kw = {"swiglu": kind == "down", "norm": norms[0] if normed else None}
            x = torch.randn((m, projs[0].k * (2 if kind == "down" else 1)),
                            generator=gen, device="cuda",
                            dtype=torch.float32 if kind == "o" else bf)
            modes = ["library"]
            if m <= 128:
                modes.append("skinny")
            if m <= (8 if normed else 128):
                modes.append("fused")
            graphs = {}
            cap = torch.cuda.Stream()
            for mode in modes:
                for p in projs:
                    p.mode = mode
                # first calls (library tuning, code loading) stay outside
                # the capture
                for p in projs:
                    p(x, **kw)
                torch.cuda.synchronize()
                g = torch.cuda.CUDAGraph()
                with torch.cuda.graph(g, stream=cap):
                    for p in projs:
                        p(x, **kw)
                graphs[mode] = g
            torch.cuda.synchronize()
            times = {mode: float("inf") for mode in modes}
            for _ in range(3):
                for mode in modes:
                    e0 = torch.cuda.Event(enable_timing=True)
                    e1 = torch.cuda.Event(enable_timing=True)
                    e0.record()
                    graphs[mode].replay()
                    e1.record()
                    torch.cuda.synchronize()
                    times[mode] = min(times[mode], e0.elapsed_time(e1))
            del graphs
            best = min(times, key=times.get)
            for p in projs:
                p.mode = best
            picks[kind] = {"library": "library_gemm", "skinny": "laminar_linear",
                           "fused": "laminar_linear_fused_input"}[best]
        return picks

    stream = torch.cuda.current_stream()
    choose(1)                 # first calls load code objects: not timed
    curves = []
    for ctx in contexts:
        points = []
        for m in batches:
            picks = choose(m)
            n_tok = ctx + 1                       # cached tokens + the new one
            pages = -(-n_tok // 16)
            kp = torch.randn((m * pages, hkv, 16 * d), generator=gen,
                             device="cuda", dtype=bf)
            vp = torch.randn_like(kp)
            # pages as a paged allocator hands them out once it has seen
            # some churn: a random permutation of the pool (with each
            # trajectory's pages contiguous, every workgroup walks the pool
            # at the same stride and attention ran ~20% slower)
            table = torch.randperm(m * pages, generator=gen, device="cuda"
                                   ).to(torch.int32).view(m, pages)
            lens_host = np.full(m, n_tok, np.int32)
            lens = torch.as_tensor(lens_host, device="cuda")
            att = PagedDecodeAttention(
                batch=m, num_q_heads=hq, num_kv_heads=hkv, head_dim=d,
                num_pages=m * pages, max_blocks_per_seq=pages,
                seq_lens_host=lens_host, softmax_scale=d ** -0.5,
                q_row_stride=(hq + 2 * hkv) * d)
            out, lse = att.outputs()
            x0 = torch.randn((m, h), generator=gen, device="cuda", dtype=bf)
            # QKV's skinny call makes the KV append too (its K-split
            # reduction stores K and V from 33 rows on)
            app_args = (kv_append_desc(m, hkv, d, m * pages, pages),
                        hq * d, (hq + hkv) * d, table, lens, kp, vp)

            # Steps handed from a projection's reduction to the next
            # projection: the RMS norm after O (for gate+up) and after down
            # (for the next QKV or the LM head) unless the consumer makes it
            # on load, and SwiGLU after gate+up unless down makes it on load.
            wq0, wo0, wg0, wd0 = layers[0]
            norm_after_o = wg0.mode != "fused"
            norm_after_down = wq0.mode != "fused" and lm_head.mode != "fused"
            swiglu_after_gu = wg0.mode == "skinny" and wd0.mode != "fused"

            def step():
                cur = torch.cuda.current_stream()
                x = x0.clone()                    # the residual stream
                xn = None                         # its RMS norm, when made

                for li, (wqkv, wo, wgu, wd) in enumerate(layers):
                    qkv = wqkv(x, norm=norms[2 * li], operand=xn,
                               append=app_args)
                    # q, k and v are read in place from the fused output
                    q = qkv[:, :hq * d].view(m, hq, d)
                    if not wqkv.appended:
                        k_new = qkv[:, hq * d:(hq + hkv) * d].view(m, hkv, d)
                        v_new = qkv[:, (hq + hkv) * d:].view(m, hkv, d)
                        kv_append(k_new, v_new, table, lens, kp, vp, stream=cur)
                    att(q, kp, vp, table, lens, out, lse, stream=cur)
                    if norm_after_o:
                        x, xn = wo(out.view(m, hq * d), residual=x,
                                   next_norm=norms[2 * li + 1])
                    else:
                        x, xn = wo(out.view(m, hq * d), residual=x), None
                    if swiglu_after_gu:
                        gu, act = wgu(x, norm=norms[2 * li + 1], operand=xn,
                                      swiglu_out=True)
                    else:
                        gu, act = wgu(x, norm=norms[2 * li + 1], operand=xn), None
                    nxt = norms[2 * li + 2]        # next QKV's, or the final
                    if norm_after_down:
                        x, xn = wd(gu, residual=x, swiglu=True, operand=act,
                                   next_norm=nxt)
                    else:
                        x, xn = wd(gu, residual=x, swiglu=True, operand=act), None
                return lm_head(x, norm=norms[2 * L], operand=xn)

            # The step is ~400 launches: capture it in a HIP graph so the
            # curve shows the GPU's time, not the host's launch rate.
            side = torch.cuda.Stream()
            side.wait_stream(stream)
            with torch.cuda.stream(side):
                eager = step()
            stream.wait_stream(side)
            torch.cuda.synchronize()
            graph = torch.cuda.CUDAGraph()
            with torch.cuda.graph(graph):
                logits = step()
            graph.replay()
            torch.cuda.synchronize()
            first = logits.clone()
            graph.replay()
            torch.cuda.synchronize()
            # every replay must reproduce the eager step bit for bit
            bits = lambda t: t.view(torch.int16)
            assert bool(torch.isfinite(eager).all()), "non-finite logits"
            assert torch.equal(bits(first), bits(eager)), "graph replay differs"
            assert torch.equal(bits(logits), bits(eager)), "graph replays differ"
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            for _ in range(reps):
                graph.replay()
            e1.record(stream)
            torch.cuda.synchronize()
            ms = e0.elapsed_time(e1) / reps
            del graph, logits, eager, first
            model_ms = 1e3 * N.laminar_roofline_step_seconds(shape, m, ctx,
                                                             peak_f, peak_bw)
            points.append({"batch": m, "ms": round(ms, 3),
                           "roofline_ms": round(model_ms, 3),
                           "projections": picks})
            print(f"[latency] context {ctx} batch {m}: {ms:.3f} ms "
                  f"(roofline {model_ms:.3f} ms)", file=sys.stderr, flush=True)
            att.close()
            del kp, vp, att
            torch.cuda.empty_cache()
        base = points[0]["ms"]
        knee = next((p["batch"] for p in points if p["ms"] > 1.1 * base), None)
        curves.append({"context": ctx, "points": points,
                       "first_batch_10pct_slower_than_batch_1": knee})
    del layers, lm_head, Proj
    torch.cuda.empty_cache()
    return {"model": f"{model_name} shapes, random bf16 weights, {L} layers "
                     "+ LM head",
            "roofline_batch_bound": bound, "peak_flops": peak_f,
            "peak_bw": peak_bw, "curves": curves}


ALL_WORKLOADS = ("tiny", "7b_pre_repack", "post_repack", "32b_fp8",
                 "agentic_mix", "32b_fp8_tp4", "agentic_mix_tp8")


def host_workers() -> int:
    return max(1, len(os.sched_getaffinity(0)))


def oracle_parity(wl, out, lse):
    """Every trajectory and head of the GPU's out and lse against the fp64
    oracle on the host; returns the errors and the oracle's wall time."""
    import numpy as np
    from threadpoolctl import threadpool_limits

    from oracle import decode_attention_from_host
    from workloads import host_arrays

    o = out.cpu().numpy()
    l = lse.cpu().numpy()
    arrays = host_arrays(wl)
    cores = host_workers()
    with threadpool_limits(1):
        t0 = time.perf_counter()
        ro, rl = decode_attention_from_host(arrays, workers=cores)
        dt = time.perf_counter() - t0
    del arrays
    fin = np.isfinite(rl)
    ok_shape = (np.isfinite(o).all() and np.isfinite(l[fin]).all()
                and np.array_equal(np.isneginf(l), np.isneginf(rl)))
    eo = float(np.abs(o - ro).max()) if o.size else 0.0
    el = float(np.abs(l[fin] - rl[fin]).max()) if fin.any() else 0.0
    ok = bool(ok_shape) and eo <= PARITY_TOL and el <= PARITY_TOL
    if not ok:
        print(f"[bench] {wl.cfg.name}: parity FAILED (out {eo:.2e}, lse {el:.2e}, "
              f"rows written and finite: {bool(ok_shape)})", file=sys.stderr,
              flush=True)
    return {"max_abs_err_out": eo, "max_abs_err_lse": el,
            "all_rows_written_and_finite": bool(ok_shape),
            "within_tolerance": ok, "tolerance": PARITY_TOL,
            "trajectories_checked": int(wl.batch),
            "oracle_s": round(dt, 3), "oracle_threads": cores}


def measure(torch, N, name, steps, warm, args, seed=None):
    """One workload: `steps` timed whole steps (host plan, table upload,
    partial kernel, merge) after `warm` untimed ones; then the same with one
    plan reused (one layer's call of a decode step whose plan all layers
    share); then each kernel launched `steps` times back to back (its
    average launch duration); every region bracketed by two HIP events on
    the launch stream. Then one more whole step into NaN-filled outputs,
    checked against the oracle over every trajectory. Returns (entry,
    extras)."""
    import numpy as np

    from paper_2510_12633_amd.api import KV_DTYPES, num_cus
    from workloads import get_config, make_workload, prefix_groups

    cfg = get_config(name)
    wl = make_workload(cfg, seed=seed, device="cuda")
    dev_lens = torch.as_tensor(wl.seq_lens, device="cuda")
    bt = torch.as_tensor(wl.block_table, device="cuda")
    cus = num_cus()
    desc = N.LaminarAttnDesc(
        batch=wl.batch, num_q_heads=cfg.num_q_heads,
        num_kv_heads=cfg.num_kv_heads, head_dim=cfg.head_dim, page_size=16,
        num_pages=wl.num_pages, max_blocks_per_seq=wl.block_table.shape[1],
        kv_dtype=KV_DTYPES[cfg.kv_dtype], softmax_scale=wl.softmax_scale,
        k_scale=None if wl.k_scale is None else wl.k_scale.data_ptr(),
        v_scale=None if wl.v_scale is None else wl.v_scale.data_ptr(),
        pages_per_item=args.pages_per_item, waves_per_item=args.waves_per_item)
    lens_host = np.ascontiguousarray(wl.seq_lens, dtype=np.int32)

    kv_bytes = wl.kv_bytes_unique()
    alg_bytes = wl.algorithmic_bytes()
    rot = Rotation(wl) if kv_bytes < (1 << 30) else None

    out = torch.empty((wl.batch, cfg.num_q_heads, cfg.head_dim),
                      dtype=torch.float32, device="cuda")
    lse = torch.empty((wl.batch, cfg.num_q_heads), dtype=torch.float32,
                      device="cuda")
    stream = torch.cuda.current_stream()
    sh = stream.cuda_stream

    group_of, group_pages = prefix_groups(wl)
    use_cascade = group_of is not None and args.cascade != "off"

    def make_plan():
        if use_cascade:
            return N.laminar_plan_create_cascade(desc, lens_host, group_of,
                                                 group_pages, cus)
        return N.laminar_plan_create(desc, lens_host, cus)

    plan0 = make_plan()
    ws_bytes = N.laminar_plan_workspace_bytes(plan0)
    n_items = N.laminar_plan_num_items(plan0)
    n_merges = N.laminar_plan_num_merges(plan0)
    ppi = N.laminar_plan_pages_per_item(plan0)
    waves = N.laminar_plan_waves_per_item(plan0)
    ws = torch.empty(max(ws_bytes, 256), dtype=torch.uint8, device="cuda")
    N.laminar_plan_bind_workspace(plan0, ws, ws_bytes, sh)

    plan_ns, bind_ns = [], []
    live = [plan0]

    def one_step(i, fixed=False, partial=True, merge=True):
        if fixed:
            plan = plan0
        else:
            t0 = time.perf_counter_ns()
            plan = make_plan()
            t1 = time.perf_counter_ns()
            N.laminar_plan_bind_workspace(plan, ws, ws_bytes, sh)
            plan_ns.append(t1 - t0)
            bind_ns.append(time.perf_counter_ns() - t1)
            live.append(plan)
        kp, vp = rot.get(i) if rot else (wl.k_pages, wl.v_pages)
        if partial:
            N.laminar_decode_attn_partial(plan, wl.q, kp, vp, bt, dev_lens,
                                          out, lse, sh)
        if merge:
            N.laminar_decode_attn_merge(plan, out, lse, sh)

    def release():
        # plans are destroyed only after the stream has passed their uploads
        torch.cuda.synchronize()
        for p in live[1:]:
            N.laminar_plan_destroy(p)
        live[1:] = []

    def timed(fn):
        """`steps` calls of fn after `warm` untimed ones, bracketed by two
        HIP events on the launch stream (nothing else is recorded between
        the calls: an event per launch adds a few microseconds to each)."""
        for i in range(warm):
            fn(i)
        release()
        plan_ns.clear()
        bind_ns.clear()
        t_start = torch.cuda.Event(enable_timing=True)
        t_end = torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        wall0 = time.perf_counter()
        t_start.record(stream)
        for i in range(steps):
            fn(warm + i)
        t_end.record(stream)
        torch.cuda.synchronize()
        wall = time.perf_counter() - wall0
        return t_start.elapsed_time(t_end) / steps, wall

    # the timed region: whole steps (plan, upload, partial, merge)
    ms_step, wall = timed(lambda i: one_step(i, fixed=args.fixed_plan))
    plan_host, bind_host = list(plan_ns), list(bind_ns)
    release()
    # one layer's call with the step's plan already uploaded, then each
    # kernel launched back to back on its own (average launch duration)
    ms_layer = timed(lambda i: one_step(i, fixed=True))[0]
    k1_ms = timed(lambda i: one_step(i, fixed=True, merge=False))[0]
    k2_ms = timed(lambda i: one_step(i, fixed=True, partial=False))[0]
    plan_ns[:], bind_ns[:] = plan_host, bind_host
    release()

    step_s = ms_step / 1e3
    achieved = alg_bytes / (k1_ms / 1e3) / 1e9
    traffic, traffic_src = read_traffic(cfg.name)

    # one more whole step into NaN-filled outputs, against the oracle
    out.fill_(float("nan"))
    lse.fill_(float("nan"))
    one_step(0)
    release()
    parity = None if args.no_parity else oracle_parity(wl, out, lse)

    entry = {
        "workload": cfg.name,
        "batch": wl.batch,
        "heads_q_kv": [cfg.num_q_heads, cfg.num_kv_heads],
        "kv_dtype": cfg.kv_dtype,
        "context_tokens": int(wl.seq_lens.sum()),
        "kv_bytes": kv_bytes,
        "algorithmic_bytes": alg_bytes,
        "decode_items_us": round(k1_ms * 1e3, 2),
        "decode_merge_us": round(k2_ms * 1e3, 2),
        "step_ms": round(ms_step, 5),
        "layer_call_ms": round(ms_layer, 5),
        "kv_TBps_step": round(kv_bytes / step_s / 1e12, 4),
        "frac_hbm_peak_step": round(kv_bytes / step_s / 1e9 / HBM_PEAK_GBPS, 4),
        "frac_hbm_peak_layer_call": round(kv_bytes / (ms_layer / 1e3) / 1e9
                                          / HBM_PEAK_GBPS, 4),
        "frac_hbm_peak_kernel": round(achieved / HBM_PEAK_GBPS, 4),
        "tokens_per_s": round(wl.batch / step_s, 1),
        "traffic_over_algorithmic": (round(traffic / alg_bytes, 4)
                                     if traffic else None),
        "work_items": n_items,
        "cascade_prefix": use_cascade,
        "plan_host_us": round(sum(plan_ns) / len(plan_ns) / 1e3, 2)
        if plan_ns else None,
    }
    if parity:
        entry.update(parity)
    extras = {
        "wl": wl, "cfg": cfg, "ms_step": ms_step,
        "k1_ms": k1_ms, "k2_ms": k2_ms, "wall": wall, "achieved": achieved,
        "traffic": traffic, "traffic_src": traffic_src, "plan_ns": plan_ns,
        "bind_ns": bind_ns, "ppi": ppi, "waves": waves, "n_items": n_items,
        "n_merges": n_merges, "use_cascade": use_cascade, "rot": rot,
        "parity": parity, "ms_layer": ms_layer,
    }
    N.laminar_plan_destroy(plan0)
    del ws, out, lse
    return entry, extras


def main(argv=None):
    args = parse_args(argv)
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not "
              "supported (the decode-attention path needs no collectives and "
              "shards by trajectory or kv-head with no exchange).",
              file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2510_12633_amd import _native as N
    from workloads import get_config

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    N.lib()      # fail loudly if the HIP library is not built

    cfg = get_config(args.workload)
    print(f"[bench] {cfg.name}: {args.steps} steps after {args.warmup}",
          file=sys.stderr, flush=True)
    entry, x = measure(torch, N, cfg.name, args.steps, args.warmup, args,
                       seed=args.seed)
    wl = x["wl"]
    ms_step = x["ms_step"]
    step_s = ms_step / 1e3
    kv_bytes = wl.kv_bytes_unique()
    alg_bytes = wl.algorithmic_bytes()
    value = kv_bytes / step_s / 1e12
    roofline = {
        "bound": "hbm",
        "kernel": PARTIAL_KERNEL,
        "achieved": round(x["achieved"], 1),
        "peak": HBM_PEAK_GBPS,
        "unit": "GB/s",
        "frac": round(x["achieved"] / HBM_PEAK_GBPS, 4),
        "traffic": x["traffic"],
        "algorithmic_bytes_per_launch": alg_bytes,
        "avg_launch_ms": round(x["k1_ms"], 5),
    }
    plan_ns, bind_ns = x["plan_ns"], x["bind_ns"]
    result = {
        "metric": METRIC,
        "value": round(value, 4),
        "unit": "TB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if cfg.kv_dtype == "bf16" else "fp8e4m3-kv/bf16",
        "data": "synthetic",
        "config": {
            "workload": cfg.name,
            "batch": wl.batch,
            "q_heads": cfg.num_q_heads,
            "kv_heads": cfg.num_kv_heads,
            "head_dim": cfg.head_dim,
            "kv_dtype": cfg.kv_dtype,
            "context_tokens": int(wl.seq_lens.sum()),
            "seed": wl.seed,
            "pages_per_item": x["ppi"],
            "waves_per_item": x["waves"],
            "work_items": x["n_items"],
            "merged_units": x["n_merges"],
            "plan_every_step": not args.fixed_plan,
            "cascade_prefix": x["use_cascade"],
            "kv_pool_copies_rotated": x["rot"].n if x["rot"] else 1,
        },
        "frac_hbm_peak": round(value * 1e3 / HBM_PEAK_GBPS, 4),
        "tokens_per_s": round(wl.batch / step_s, 1),
        "context_tokens_per_s": round(float(wl.seq_lens.sum()) / step_s, 1),
        "kv_bytes": kv_bytes,
        "algorithmic_bytes": alg_bytes,
        "kernel_ms": {"decode_items": round(x["k1_ms"], 5),
                      "decode_merge": round(x["k2_ms"], 5)},
        "kernel_timing": "average launch duration: the same plan's kernel "
                         f"launched {args.steps} times back to back between "
                         "two HIP events on the launch stream",
        # one layer's call with the step's plan already uploaded (every
        # layer of a decode step shares one plan)
        "layer_call_ms": round(x["ms_layer"], 5),
        "plan_host_ms": round(sum(plan_ns) / max(len(plan_ns), 1) / 1e6, 5)
        if plan_ns else None,
        # bind: tables into a pinned staging slot and the upload launch; it
        # waits when the host is eight steps ahead of the GPU
        "bind_host_ms": round(sum(bind_ns) / max(len(bind_ns), 1) / 1e6, 5)
        if bind_ns else None,
        "wall_s_timed": round(x["wall"], 4),
        "roofline": roofline,
    }
    if x["parity"]:
        result["max_abs_err_out"] = x["parity"]["max_abs_err_out"]
        result["max_abs_err_lse"] = x["parity"]["max_abs_err_lse"]
        result["parity"] = x["parity"]
    if x["traffic_src"] == "stale":
        result["roofline"]["traffic_note"] = "counters predate the current kernel"
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(wl, args.cpu_budget_s)
    del x, wl
    torch.cuda.empty_cache()
    if not args.no_calibrate:
        cal = calibrate(torch, N)
        result["hbm_calibration_GBps"] = {k: round(v, 1) for k, v in cal.items()}
        result["frac_of_calibrated_read"] = round(value * 1e3 / cal["read"], 4)
        result["frac_of_calibrated_gather"] = round(
            roofline["achieved"] / cal["gather_4KiB"], 4)
        # the fixed cost of a kernel in a captured graph (the decode-step
        # curve's floor per launch)
        result["graph_launch_floor_us"] = graph_launch_floor(torch)
    if not args.no_per_config:
        rows = []
        for name in ALL_WORKLOADS:
            if name == cfg.name:
                rows.append(entry)
                continue
            print(f"[bench] per-config {name}", file=sys.stderr, flush=True)
            e, xx = measure(torch, N, name, args.steps, args.warmup, args)
            del xx
            torch.cuda.empty_cache()
            rows.append(e)
        result["per_config"] = rows
    else:
        result["per_config"] = [entry]
    if not (args.no_append and args.no_repack):
        from workloads import make_workload
        wl = make_workload(cfg, seed=args.seed, device="cuda")
        if not args.no_append:
            app = measure_append(torch, wl)
            if app is not None:
                result["kv_append"] = app
        if not args.no_repack:
            result["repack"] = measure_repack(torch, N, wl)
        del wl
        torch.cuda.empty_cache()
    if not args.no_projections:
        result["projections"] = measure_projections(torch, N)
    if args.latency_curve:
        kw = {"model": args.curve_model}
        if args.curve_batches:
            kw["batches"] = tuple(int(x) for x in args.curve_batches.split(","))
        if args.curve_contexts:
            kw["contexts"] = tuple(int(x) for x in args.curve_contexts.split(","))
        result["latency_curve"] = latency_curve(torch, N, **kw)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
