#!/usr/bin/env python3
"""Benchmark of the BF1 prefill forward on one MI355X.

    python bench.py [--steps K] [--warmup W] [--workload NAME] [--sweep]

A step is one pass of the whole hot path over one batch of synthetic input
already resident in HBM: the route planner writes the CSR table, then the
attention kernel walks it (bf1_plan + bf1_attn_fwd_csr on one stream).  The
timed region is exactly K steps bracketed by device synchronisation.  The
default workload is the Qwen3-0.6B layer geometry at n = 32768 (batch 1,
16 q-heads, 8 kv-heads, head_dim 128, block width 64, two local blocks).

The last line of stdout is one JSON record:
  value      selected-interaction TFLOP/s of the whole step
             (4 * head_dim * selected pairs * Hq * batch / step time)
  roofline   the attention kernel alone: achieved TFLOP/s (HIP events on its
             stream, averaged over the K timed launches) against the
             published dense bf16 MFMA peak of MI355X (2.5 PFLOP/s)
  mfma_reference  what a tuned library GEMM reaches on this chip: PyTorch's
             bf16 matmul (hipBLASLt) at 8192^3 with N(0,1) operands and with
             all-zero operands.  The chip's clock is held by its power limit,
             and the matrix cores draw more power on random data, so the
             sustainable bf16 rate on random operands sits well below the
             published peak; the attention kernel's rate is given against it
  dense      the in-house dense causal kernel timed with the paper's
             protocol (5 warmups, 30 reps, two opposite orders, median of the
             two order medians, §4.3) next to BF1 timed the same way; PyTorch's
             own scaled_dot_product_attention (the "native SDPA" the paper
             compares against; flash backend only, K/V heads expanded to the
             query heads) timed beside them
  backward   the backward (dQ, dK, dV) of the same layer, timed with the
             same two-order protocol next to the forward: one bf1_attn_bwd
             call (Delta, dQ, dK/dV and the partial-sum reduce) per rep,
             algorithmic TFLOP/s = 10 * head_dim * selected pairs * Hq * batch
             / time, against the same bf16 MFMA peak
  route_variants  the same kernel (bf1_attn_fwd_csr) over BF1's table and
             the two equal-pair-count controls of §4.3 / §5.1 (matched local
             sliding, static random graph seed 17), timed with the paper
             protocol extended to three routes (orders A,B,C then C,B,A),
             each with its communication depth (§5.2)
  decode     one-token decode over a paged cache (§5.4, Table 3): contexts
             32K / 64K, batch 1 / 8 / 32, a plan per route epoch; the step
             (split + merge kernels) and the planner timed as replayed HIP
             graphs (device time, as a serving loop runs them) and eagerly
             (host launch included); the dense decode through the same
             kernels next to it; achieved HBM GB/s on the algorithmic bytes
             (the K/V rows each token reads, its query and output)
  ttft       whole-model prefill of the Qwen3-0.6B geometry with random
             weights (§4.3, §5.3): warm time to first token at 8K / 16K / 32K
             with every attention layer dense, the middle eight on the BF1
             route, and all 28 on the BF1 route (timing only)
  sweep      the length sweep n = 1K..64K for block widths 64 and 128 (the
             metric's range): BF1 and the in-house dense kernel per point,
             timed two ways with the two-order protocol -- calls captured in a
             HIP graph and replayed (no host launch cost, which dominates
             short lengths, but graph nodes add a few microseconds between
             kernels) and events around each host call (kernel time plus any
             launch gap).  Both bound the kernel's device time from above;
             device_ms is the smaller.  % of the bf16 MFMA peak and the
             BF1/dense speedup follow from device_ms.
  cpu_baseline  the fp64 CPU oracle on a bounded sample of the workload
  cpu_baseline_configs  the same oracle on the tiny (n=512), n=4096 and
             n=30001 batch-2 peaked workloads

--sweep additionally times n = 1K..64K for block widths 64 and 128 with the
two-order protocol and writes one JSON record per point to --sweep-out.

--load KIND --load-seconds S runs one workload back to back for S seconds
and prints its time per call, nothing else (for sampling the GPU's shader
clock from another process while it runs): attn (the BF1 forward of the
default workload), attn_q0 (the same with Q = 0), dense (the in-house dense
causal kernel on the same inputs), bwd (the backward of the BF1 forward on
the same inputs), gemm / gemm_zero (the
8192^3 bf16 matmul of mfma_reference on N(0,1) / all-zero operands).
"""

import argparse
import json
import os
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0   # MI355X published dense bf16 MFMA peak
PEAK_HBM_GBS = 8000.0


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=30)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="qwen_n32768")
    ap.add_argument("--reps", type=int, default=30, help="reps per order in the two-order protocol")
    ap.add_argument("--sweep", action="store_true")
    ap.add_argument("--sweep-out", default="sweep.jsonl")
    ap.add_argument("--no-dense", action="store_true")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-backward", action="store_true")
    ap.add_argument("--no-variants", action="store_true")
    ap.add_argument("--no-decode", action="store_true")
    ap.add_argument("--no-ttft", action="store_true")
    ap.add_argument("--no-gemm-ref", action="store_true")
    ap.add_argument("--load", choices=["attn", "attn_q0", "dense", "bwd", "gemm", "gemm_zero"], default=None,
                    help="run one workload back to back (see the module docstring) and exit")
    ap.add_argument("--load-seconds", type=float, default=8.0)
    ap.add_argument("--no-sweep-device", action="store_true",
                    help="skip the default 1K-64K device-time sweep")
    ap.add_argument("--cpu-seconds", type=float, default=15.0,
                    help="time bound of the CPU oracle sample")
    ap.add_argument("--calib-copy-mb", type=int, default=0,
                    help="after timing, run one plain device copy of this many MiB (the "
                         "reference for scaling HBM byte counters)")
    ap.add_argument("--spinup-ms", type=float, default=200.0,
                    help="untimed attention launches before the warmup steps so the GPU "
                         "clocks have ramped up")
    ap.add_argument("--traffic-json", default=os.path.join(ROOT, "profiles", "bf1_fwd_traffic.json"))
    return ap.parse_args()


def kernel_source_hash():
    """sha256 over the forward kernel's sources (the kernel file and the
    device helpers it includes, in that order)."""
    import hashlib
    h = hashlib.sha256()
    for name in ("bf1_kernels.hip", "bf1_device.h"):
        h.update(open(os.path.join(ROOT, "paper_2608_20427_amd", "csrc", name), "rb").read())
    return h.hexdigest()


def timed_reps(torch, fn, warmup, reps):
    """Per-launch device times (ms) of fn on the current stream."""
    for _ in range(warmup):
        fn()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(reps)]
    for a, b in ev:
        a.record()
        fn()
        b.record()
    torch.cuda.synchronize()
    return [a.elapsed_time(b) for a, b in ev]


def two_order(torch, fa, fb, warmup, reps):
    """Paper protocol (§4.3): both orders, median of the two order medians."""
    a1 = timed_reps(torch, fa, warmup, reps)
    b1 = timed_reps(torch, fb, warmup, reps)
    b2 = timed_reps(torch, fb, warmup, reps)
    a2 = timed_reps(torch, fa, warmup, reps)

    def summ(x, y):
        allv = sorted(x + y)
        return {"ms": statistics.median([statistics.median(x), statistics.median(y)]),
                "p10": allv[int(0.1 * (len(allv) - 1))], "p90": allv[int(0.9 * (len(allv) - 1))]}
    return summ(a1, a2), summ(b1, b2)


def cpu_model():
    """The host CPU's model name (Linux /proc/cpuinfo), or "unknown"."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(w, max_seconds, min_seconds=0.0):
    """The fp64 oracle on a bounded sample of the workload: query blocks in
    an evenly spread order (heaviest first), 16 at a time, until the time
    bound is reached; a workload finished before min_seconds is run again,
    whole passes, until that much time has gone by."""
    from oracle import bf1_oracle as orc
    from paper_2608_20427_amd import synth
    q, k, v = synth.make_qkv(w)
    qd, kd, vd = synth.to_f64(q), synth.to_f64(k), synth.to_f64(v)
    NB = orc.num_blocks(w.n, w.b)
    order = []
    for stride_off in range(8):
        order.extend(range(NB - 1 - stride_off, -1, -8))
    rp, ci = orc.csr(w.n, w.b, w.L)
    done, passes = [], 0
    t0 = time.perf_counter()
    while True:
        for at in range(0, len(order), 16):
            chunk = order[at:at + 16]
            orc.attn_gathered_fp64(qd, kd, vd, w.b, w.L, blocks=chunk)
            done.extend(chunk)
            if time.perf_counter() - t0 > max_seconds:
                break
        else:
            passes += 1
            if time.perf_counter() - t0 < min_seconds:
                continue
        break
    dt = time.perf_counter() - t0
    pairs_of = {}
    for j in set(done):
        rows = min((j + 1) * w.b, w.n) - j * w.b
        earlier = sum(min((int(i) + 1) * w.b, w.n) - int(i) * w.b
                      for i in ci[rp[j]:rp[j + 1]] if int(i) < j)
        pairs_of[j] = rows * earlier + rows * (rows + 1) // 2
    pairs = sum(pairs_of[j] for j in done)
    flops = 4 * w.d * int(pairs) * w.Hq * w.batch
    cores = len(os.sched_getaffinity(0))
    if passes:
        what = f"the whole workload ({NB} query blocks) {passes} time(s) over"
        if len(done) > passes * NB:
            what += f" plus {len(done) - passes * NB} blocks of another pass"
    else:
        what = f"{len(done)} of {NB} query blocks (strided order, heaviest first)"
    return {"value": flops / dt / 1e12, "unit": "TFLOP/s", "cores": cores, "kind": "oracle",
            "cpu_model": cpu_model(), "seconds": dt, "gflop": flops / 1e9, "passes": passes,
            "sample": f"{what}, all {w.Hq} q-heads, batch {w.batch}, workload {w.name}; "
                      f"time bound {max_seconds:.0f} s, whole passes repeated to at least "
                      f"{min_seconds:.0f} s; fp64 NumPy gathered oracle, BLAS threads = host cores"}


def gemm_reference(torch, achieved, N=8192):
    """bf16 GEMM rate of the platform library (torch.matmul -> hipBLASLt) on
    random and on all-zero operands: the matrix cores' sustainable rate on
    random data under the chip's power limit, for reading the roofline
    fraction (the fraction itself stays against the published peak)."""
    g = torch.Generator(device="cuda")
    g.manual_seed(0)
    a = torch.randn(N, N, dtype=torch.bfloat16, device="cuda", generator=g)
    b = torch.randn(N, N, dtype=torch.bfloat16, device="cuda", generator=g)
    z = torch.zeros_like(a)
    c = torch.empty_like(a)
    flops = 2.0 * N ** 3
    out = {"what": f"torch.matmul bf16 {N}x{N}x{N} (hipBLASLt), median of 20 calls after 10 warm-up calls"}
    for name, x, y in (("random", a, b), ("zeros", z, z)):
        ms = statistics.median(timed_reps(torch, lambda: torch.matmul(x, y, out=c), 10, 20))
        out[f"{name}_tflops"] = flops / (ms * 1e-3) / 1e12
    out["random_frac_of_peak"] = out["random_tflops"] / PEAK_BF16_TFLOPS
    out["attention_over_random_gemm"] = achieved / out["random_tflops"]
    del a, b, z, c
    return out


def run_load(torch, bf1, synth, kind, seconds, workload):
    """One workload back to back for `seconds` (the --load mode): prints the
    number of calls and the device time per call."""
    if kind.startswith("attn") or kind in ("dense", "bwd"):
        w = synth.WORKLOADS[workload]
        q, k, v = synth.make_qkv(w, device="cuda")
        if kind == "attn_q0":
            q.zero_()
        o = torch.empty_like(q)
        lse = torch.empty((w.batch, w.Hq, w.n), dtype=torch.float32, device="cuda")
        rp, ci = bf1.plan(w.n, w.b, w.L)
        fn = lambda: bf1.attn_fwd_csr(q, k, v, w.b, rp, ci, out=o, lse=lse)
        if kind == "dense":
            fn = lambda: bf1.dense_causal_fwd(q, k, v, out=o, lse=lse)
        elif kind == "bwd":
            fn()
            do = synth.make_grad_out(w, device="cuda")
            dq = torch.empty(q.shape, dtype=torch.float32, device="cuda")
            dk = torch.empty(k.shape, dtype=torch.float32, device="cuda")
            dv = torch.empty_like(dk)
            ws = torch.empty(bf1.bwd_workspace_size(w.batch, w.n, w.Hq, w.Hkv, w.d, w.b, w.L),
                             dtype=torch.uint8, device="cuda")
            fn = lambda: bf1.attn_bwd(q, k, v, o, do, lse, w.b, w.L, dq=dq, dk=dk, dv=dv, workspace=ws)
    else:
        N = 8192
        g = torch.Generator(device="cuda")
        g.manual_seed(0)
        a = torch.randn(N, N, dtype=torch.bfloat16, device="cuda", generator=g)
        b = torch.randn(N, N, dtype=torch.bfloat16, device="cuda", generator=g)
        if kind == "gemm_zero":
            a.zero_()
            b.zero_()
        c = torch.empty_like(a)
        fn = lambda: torch.matmul(a, b, out=c)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    calls = 0
    t0 = time.perf_counter()
    e0.record()
    while time.perf_counter() - t0 < seconds:
        for _ in range(20):
            fn()
        calls += 20
        torch.cuda.synchronize()
    e1.record()
    torch.cuda.synchronize()
    print(f"load {kind}: {calls} calls, {e0.elapsed_time(e1) / calls * 1e3:.1f} us per call", flush=True)


def sdpa_fn(torch, q, k, v):
    """PyTorch's scaled_dot_product_attention (causal) restricted to its flash
    backend, with K/V expanded to the query heads; None where that backend is
    not available (its fallback paths are never used)."""
    from torch.nn.attention import sdpa_kernel, SDPBackend
    G = q.shape[1] // k.shape[1]
    ke = k.repeat_interleave(G, dim=1).contiguous()
    ve = v.repeat_interleave(G, dim=1).contiguous()

    def f():
        with sdpa_kernel([SDPBackend.FLASH_ATTENTION]):
            return torch.nn.functional.scaled_dot_product_attention(q, ke, ve, is_causal=True)
    try:
        f()
        torch.cuda.synchronize()
    except RuntimeError as e:
        log(f"SDPA flash backend unavailable: {str(e)[:120]}")
        return None
    return f


def run_point(torch, bf1, w, q, k, v, warmup, reps, with_dense=True):
    """Two-order timing of BF1 and dense on one workload."""
    o = torch.empty_like(q)
    lse = torch.empty((w.batch, w.Hq, w.n), dtype=torch.float32, device="cuda")
    rp, ci = bf1.plan(w.n, w.b, w.L)
    f_bf1 = lambda: bf1.attn_fwd_csr(q, k, v, w.b, rp, ci, out=o, lse=lse)
    f_dense = lambda: bf1.dense_causal_fwd(q, k, v, out=o, lse=lse)
    flops = bf1.selected_flops(w.batch, w.n, w.Hq, w.d, w.b, w.L)
    dense_flops = 4 * w.d * (w.n * (w.n + 1) // 2) * w.Hq * w.batch
    plan_ms = statistics.median(timed_reps(torch, lambda: bf1.plan(w.n, w.b, w.L, rp, ci), 3, 20))
    if with_dense:
        sb, sd = two_order(torch, f_bf1, f_dense, warmup, reps)
    else:
        x = timed_reps(torch, f_bf1, warmup, reps)
        sb, sd = {"ms": statistics.median(x), "p10": min(x), "p90": max(x)}, None
    rec = {"workload": w.name, "n": w.n, "b": w.b, "L": w.L, "batch": w.batch, "Hq": w.Hq,
           "Hkv": w.Hkv, "head_dim": w.d, "selected_gflop": flops / 1e9,
           "bf1_ms": sb["ms"], "bf1_p10_ms": sb["p10"], "bf1_p90_ms": sb["p90"],
           "bf1_tflops": flops / sb["ms"] / 1e9,
           "bf1_pct_peak": 100 * flops / sb["ms"] / 1e9 / PEAK_BF16_TFLOPS,
           "plan_us": plan_ms * 1e3}
    if sd is not None:
        rec.update({"dense_gflop": dense_flops / 1e9, "dense_ms": sd["ms"], "dense_p10_ms": sd["p10"],
                    "dense_p90_ms": sd["p90"], "dense_tflops": dense_flops / sd["ms"] / 1e9,
                    "dense_pct_peak": 100 * dense_flops / sd["ms"] / 1e9 / PEAK_BF16_TFLOPS,
                    "speedup_vs_dense": sd["ms"] / sb["ms"],
                    "pair_reduction": dense_flops / flops})
        f_sdpa = sdpa_fn(torch, q, k, v)
        if f_sdpa is not None:
            _, ss = two_order(torch, f_bf1, f_sdpa, warmup, reps)
            rec.update({"sdpa_ms": ss["ms"], "sdpa_tflops": dense_flops / ss["ms"] / 1e9,
                        "speedup_vs_sdpa": ss["ms"] / sb["ms"]})
            del f_sdpa
    return rec


def graph_reps(torch, fn, inner, reps):
    """Device time per call of fn (ms, one value per replay): `inner` calls
    captured in one HIP graph on a side stream, the graph replayed `reps`
    times with events around each replay."""
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        fn()
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        for _ in range(inner):
            fn()
    g.replay()
    torch.cuda.synchronize()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(reps)]
    for a, b in ev:
        a.record()
        g.replay()
        b.record()
    torch.cuda.synchronize()
    out = [a.elapsed_time(b) / inner for a, b in ev]
    del g
    return out


def sweep_device(torch, bf1, synth, reps=8):
    """The 1K..64K sweep for b = 64 and 128: per point BF1 and dense device
    time (graph replay) and per-call time, each in both orders (median of the
    two order medians)."""
    out = []
    for w64, w128 in zip(synth.sweep(64), synth.sweep(128)):
        q, k, v = synth.make_qkv(w64, device="cuda")     # the two sweeps share inputs (same seed)
        o = torch.empty_like(q)
        lse = torch.empty((1, w64.Hq, w64.n), dtype=torch.float32, device="cuda")
        f_dense = lambda: bf1.dense_causal_fwd(q, k, v, out=o, lse=lse)
        dense_flops = 4 * w64.d * (w64.n * (w64.n + 1) // 2) * w64.Hq * w64.batch
        for w in (w64, w128):
            rp, ci = bf1.plan(w.n, w.b, w.L)
            f_bf1 = lambda: bf1.attn_fwd_csr(q, k, v, w.b, rp, ci, out=o, lse=lse)
            flops = bf1.selected_flops(w.batch, w.n, w.Hq, w.d, w.b, w.L)
            inner_d = max(1, min(16, (1 << 16) // w.n * 2))
            a1 = graph_reps(torch, f_bf1, 16, reps)
            d1 = graph_reps(torch, f_dense, inner_d, reps)
            d2 = graph_reps(torch, f_dense, inner_d, reps)
            a2 = graph_reps(torch, f_bf1, 16, reps)
            med = lambda x, y: statistics.median([statistics.median(x), statistics.median(y)])
            gb, gd = med(a1, a2), med(d1, d2)
            cb, cd = two_order(torch, f_bf1, f_dense, 3, 10)
            bd, dd = min(gb, cb["ms"]), min(gd, cd["ms"])
            plan_ms = statistics.median(graph_reps(torch, lambda: bf1.plan(w.n, w.b, w.L, rp, ci), 16, 4))
            rec = {"n": w.n, "b": w.b, "L": w.L, "Hq": w.Hq, "Hkv": w.Hkv, "head_dim": w.d, "seed": w.seed,
                   "selected_gflop": flops / 1e9, "dense_gflop": dense_flops / 1e9,
                   "bf1_device_ms": bd, "bf1_device_tflops": flops / bd / 1e9,
                   "bf1_device_pct_peak": 100 * flops / bd / 1e9 / PEAK_BF16_TFLOPS,
                   "dense_device_ms": dd, "dense_device_tflops": dense_flops / dd / 1e9,
                   "dense_device_pct_peak": 100 * dense_flops / dd / 1e9 / PEAK_BF16_TFLOPS,
                   "speedup_device": dd / bd,
                   "bf1_graph_ms": gb, "dense_graph_ms": gd,
                   "bf1_call_ms": cb["ms"], "dense_call_ms": cd["ms"], "speedup_call": cd["ms"] / cb["ms"],
                   "plan_device_us": plan_ms * 1e3, "pair_reduction": dense_flops / flops}
            out.append(rec)
            log(f"sweep n={w.n} b={w.b}: bf1 {bd * 1e3:.1f} us device ({rec['bf1_device_pct_peak']:.1f}% of peak;"
                f" graph {gb * 1e3:.1f}, per call {cb['ms'] * 1e3:.1f}); dense {dd * 1e3:.1f} us device "
                f"({rec['dense_device_pct_peak']:.1f}%); speedup {dd / bd:.2f}x device, "
                f"{cd['ms'] / cb['ms']:.2f}x per call; plan {plan_ms * 1e3:.1f} us")
            del rp, ci
        del q, k, v, o, lse
        torch.cuda.empty_cache()
    return out


def backward_point(torch, bf1, synth, w, q, k, v, warmup, reps):
    """Two-order timing of the backward against the forward on one workload;
    o and lse come from the forward, dO from the seeded generator."""
    o, lse = bf1.attn_fwd(q, k, v, w.b, w.L)
    do = synth.make_grad_out(w, device="cuda")
    dq = torch.empty(q.shape, dtype=torch.float32, device="cuda")
    dk = torch.empty(k.shape, dtype=torch.float32, device="cuda")
    dv = torch.empty(v.shape, dtype=torch.float32, device="cuda")
    ws = torch.empty(bf1.bwd_workspace_size(w.batch, w.n, w.Hq, w.Hkv, w.d, w.b, w.L),
                     dtype=torch.uint8, device="cuda")
    f_bwd = lambda: bf1.attn_bwd(q, k, v, o, do, lse, w.b, w.L, dq=dq, dk=dk, dv=dv, workspace=ws)
    f_fwd = lambda: bf1.attn_fwd(q, k, v, w.b, w.L, out=o, lse=lse)
    sf, sb = two_order(torch, f_fwd, f_bwd, warmup, reps)
    flops = bf1.selected_bwd_flops(w.batch, w.n, w.Hq, w.d, w.b, w.L)
    tf = flops / sb["ms"] / 1e9
    return {"workload": w.name, "bwd_ms": sb["ms"], "bwd_p10_ms": sb["p10"], "bwd_p90_ms": sb["p90"],
            "fwd_ms": sf["ms"], "bwd_over_fwd": sb["ms"] / sf["ms"],
            "bwd_algorithmic_gflop": flops / 1e9, "bwd_tflops": tf,
            "bwd_pct_peak": 100 * tf / PEAK_BF16_TFLOPS,
            "workspace_mb": ws.numel() / 1e6,
            "kernels": "D and LSE log2 e (bwd_delta_kernel), dK/dV and dS (bwd_dkdv_kernel), "
                       "partial reduce (bwd_reduce_kernel), dQ from dS (bwd_dq_kernel); "
                       "per-kernel times are in the rocprofv3 summary"}


def variants_point(torch, bf1, w, q, k, v, warmup, reps):
    """BF1, matched sliding and static-random tables through the CSR kernel:
    every table has BF1's pair count, so equal times mean cost tracks pairs
    and not topology (§5.1)."""
    o = torch.empty_like(q)
    lse = torch.empty((w.batch, w.Hq, w.n), dtype=torch.float32, device="cuda")
    kinds = ["bf1", "sliding", "static_random"]
    tables, depth = {}, {}
    for kd in kinds:
        rp, ci = bf1.plan_variant(kd, w.n, w.b, w.L, 17)
        depth[kd] = bf1.route_depth(rp, ci) if len(rp) - 1 <= 16384 else None
        tables[kd] = (torch.from_numpy(rp).cuda(), torch.from_numpy(ci).cuda())
    fns = {kd: (lambda t=tables[kd]: bf1.attn_fwd_csr(q, k, v, w.b, t[0], t[1], out=o, lse=lse))
           for kd in kinds}
    runs = {kd: [] for kd in kinds}
    for order in (kinds, kinds[::-1]):
        for kd in order:
            runs[kd].append(timed_reps(torch, fns[kd], warmup, reps))
    flops = bf1.selected_flops(w.batch, w.n, w.Hq, w.d, w.b, w.L)
    out = {"workload": w.name, "seed": 17, "selected_gflop": flops / 1e9}
    for kd in kinds:
        ms = statistics.median([statistics.median(x) for x in runs[kd]])
        out[kd] = {"ms": ms, "tflops": flops / ms / 1e9, "max_shortest_path": depth[kd]}
    for kd in kinds[1:]:
        out[kd]["time_vs_bf1"] = out[kd]["ms"] / out["bf1"]["ms"]
    return out


def graph_ms(torch, fn, replays, inner=32):
    """Device time per call of fn: `inner` calls captured in one HIP graph,
    the graph replayed back to back; host launch cost is paid once per
    replay and spread over the inner calls."""
    fn()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        for _ in range(inner):
            fn()
    for _ in range(2):
        g.replay()
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(replays):
        g.replay()
    b.record()
    torch.cuda.synchronize()
    return a.elapsed_time(b) / (replays * inner)


def decode_point(torch, bf1, synth, w, reps):
    """BF1 and dense decode steps over the same paged cache."""
    q, kp, vp, sl, table, num_pages = synth.make_decode_device(w)
    o = torch.empty_like(q)
    lse = torch.empty((w.batch, w.Hq), dtype=torch.float32, device="cuda")
    rec = {"workload": w.name, "batch": w.batch, "context": w.ctx, "Hq": w.Hq, "Hkv": w.Hkv,
           "head_dim": w.d, "block_width": w.b, "local_blocks": w.L}
    for dense in (False, True):
        stride = bf1.decode_plan_stride(w.ctx, w.b, w.L, dense)
        plan = bf1.decode_plan(sl, table, num_pages, stride, w.b, w.L, dense)
        ws = torch.empty(max(16, bf1.decode_workspace_size(w.batch, w.Hq, w.Hkv, w.d, stride)),
                         dtype=torch.uint8, device="cuda")
        step = lambda: bf1.attn_decode(q, kp, vp, sl, plan, w.b, out=o, lse=lse, workspace=ws)
        mkplan = lambda: bf1.decode_plan(sl, table, num_pages, stride, w.b, w.L, dense, plan=plan)
        step_graph = graph_ms(torch, step, 10)
        plan_graph = graph_ms(torch, mkplan, 10)
        step_eager = statistics.median(timed_reps(torch, step, 5, reps))
        plan_eager = statistics.median(timed_reps(torch, mkplan, 5, reps))
        torch.cuda.synchronize()
        counts = plan[:, 1].cpu().tolist()
        keys = sum((int(n) - 1) % w.b + 1 + w.b * int(c) for n, c in zip(sl.cpu().tolist(), counts))
        nbytes = keys * w.Hkv * w.d * 2 * 2 + w.batch * w.Hq * w.d * 2 * 2 + w.batch * w.Hq * 4
        key = "dense" if dense else "bf1"
        rec[key] = {"step_us_graph": step_graph * 1e3, "step_us_eager": step_eager * 1e3,
                    "plan_us_graph": plan_graph * 1e3, "plan_us_eager": plan_eager * 1e3,
                    "pages_per_token": (sum(counts) + w.batch) / w.batch,
                    "bytes_per_step": nbytes,
                    "achieved_GBs": nbytes / (step_graph * 1e-3) / 1e9,
                    "hbm_frac": nbytes / (step_graph * 1e-3) / 1e9 / PEAK_HBM_GBS,
                    "effective_us_plan_every_step": (step_graph + plan_graph) * 1e3,
                    "effective_us_plan_per_epoch": (step_graph + plan_graph / w.b) * 1e3}
        del ws, plan
    rec["speedup_vs_dense_graph"] = rec["dense"]["step_us_graph"] / rec["bf1"]["step_us_graph"]
    del q, kp, vp
    torch.cuda.empty_cache()
    return rec


def ttft_point(torch, synth, reps=5, warmup=2):
    """Warm time to first token of the decoder stack, per context and
    attention configuration (median of `reps` timed prefills)."""
    from paper_2608_20427_amd.prefill_model import PrefillStack, middle_layers
    cfg = synth.QWEN3_06B
    st = PrefillStack(cfg, synth.make_model_weights(cfg, 6000, device="cuda"))
    conds = {"dense": set(), "bf1_middle8": middle_layers(cfg, 8), "bf1_all": set(range(cfg.layers)),
             "sdpa_dense": set(), "sdpa_bf1_middle8": middle_layers(cfg, 8)}
    from torch.nn.attention import sdpa_kernel, SDPBackend

    def sdpa(Q, K, V):
        G = Q.shape[1] // K.shape[1]
        with sdpa_kernel([SDPBackend.FLASH_ATTENTION]):
            return torch.nn.functional.scaled_dot_product_attention(
                Q, K.repeat_interleave(G, dim=1), V.repeat_interleave(G, dim=1), is_causal=True)
    probe = torch.zeros((1, 2, 64, 128), dtype=torch.bfloat16, device="cuda")
    try:
        sdpa(probe, probe[:, :1].contiguous(), probe[:, :1].contiguous())
        torch.cuda.synchronize()
    except RuntimeError:
        conds.pop("sdpa_dense")
        conds.pop("sdpa_bf1_middle8")
    out = {"model": "Qwen3-0.6B geometry, random weights", "bf1_middle8_layers": sorted(conds["bf1_middle8"]),
           "contexts": {}}
    for n in (8192, 16384, 32768):
        ids = torch.from_numpy(synth.make_tokens(cfg, n, 6001)).cuda()
        rec = {}
        for name, sel in conds.items():
            dfn = sdpa if name.startswith("sdpa") else None
            for _ in range(warmup):
                st.last_logits(ids, sel, dfn)
            torch.cuda.synchronize()
            ts = []
            for _ in range(reps):
                t0 = time.perf_counter()
                st.last_logits(ids, sel, dfn)
                torch.cuda.synchronize()
                ts.append((time.perf_counter() - t0) * 1e3)
            rec[name + "_ms"] = statistics.median(ts)
        rec["speedup_middle8"] = rec["dense_ms"] / rec["bf1_middle8_ms"]
        rec["speedup_all"] = rec["dense_ms"] / rec["bf1_all_ms"]
        if "sdpa_dense_ms" in rec:
            rec["speedup_middle8_vs_sdpa_dense"] = rec["sdpa_dense_ms"] / rec["sdpa_bf1_middle8_ms"]
            rec["speedup_all_vs_sdpa_dense"] = rec["sdpa_dense_ms"] / rec["bf1_all_ms"]
        out["contexts"][str(n)] = rec
        del ids
    del st
    torch.cuda.empty_cache()
    return out


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only: the library has no multi-GPU path "
              f"(asked for --gpus {args.gpus}); run with --gpus 1", file=sys.stderr)
        sys.exit(2)
    import torch
    import paper_2608_20427_amd as bf1
    from paper_2608_20427_amd import synth

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    bf1.load()
    if args.load is not None:
        run_load(torch, bf1, synth, args.load, args.load_seconds, args.workload)
        return
    w = synth.WORKLOADS[args.workload]
    props = torch.cuda.get_device_properties(0)
    log(f"device {props.name} CUs={props.multi_processor_count}; workload {w}")
    q, k, v = synth.make_qkv(w, device="cuda")
    NB, nnz, pairs = bf1.plan_size(w.n, w.b, w.L)
    rp = torch.empty(NB + 1, dtype=torch.int32, device="cuda")
    ci = torch.empty(nnz, dtype=torch.int32, device="cuda")
    o = torch.empty_like(q)
    lse = torch.empty((w.batch, w.Hq, w.n), dtype=torch.float32, device="cuda")
    flops = bf1.selected_flops(w.batch, w.n, w.Hq, w.d, w.b, w.L)

    def plan():
        bf1.plan(w.n, w.b, w.L, rp, ci)

    def attn():
        bf1.attn_fwd_csr(q, k, v, w.b, rp, ci, out=o, lse=lse)

    # clock spin-up (untimed, on a valid route table), then the W warmup steps
    plan()
    torch.cuda.synchronize()
    t_spin = time.perf_counter()
    while (time.perf_counter() - t_spin) * 1e3 < args.spinup_ms:
        attn()
        torch.cuda.synchronize()
    for _ in range(args.warmup):
        plan()
        attn()
    torch.cuda.synchronize()
    log(f"warmup done ({args.warmup} steps)")

    # ---- timed region: exactly K steps -------------------------------------
    marks = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
             for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for a, b in marks:
        plan()
        a.record()
        attn()
        b.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    kern_ms = [a.elapsed_time(b) for a, b in marks]
    ms_per_step = wall * 1e3 / args.steps
    attn_ms = statistics.mean(kern_ms)
    log(f"timed {args.steps} steps: {ms_per_step:.4f} ms/step, attention kernel {attn_ms:.4f} ms")

    achieved = flops / (attn_ms * 1e-3) / 1e12
    # HBM bytes per launch from the committed counter summary, valid only for
    # the kernel source it was measured on (null once the kernel changed).
    traffic = None
    if os.path.exists(args.traffic_json):
        try:
            t = json.load(open(args.traffic_json))
            if t.get("workload") == w.name and t.get("kernel_source_sha256") == kernel_source_hash():
                traffic = t.get("bytes_per_launch")
        except (OSError, ValueError):
            traffic = None
    rec = {
        "metric": "BF1 prefill per-layer ms and selected-pair TFLOP/s (% MFMA peak) vs dense, 1K-64K",
        "value": flops / (ms_per_step * 1e-3) / 1e12,
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": w.name, "batch": w.batch, "seq_len": w.n, "Hq": w.Hq, "Hkv": w.Hkv,
                   "head_dim": w.d, "block_width": w.b, "local_blocks": w.L,
                   "parallelism": "none (one GPU)"},
        "per_layer_ms": ms_per_step,
        "selected_gflop": flops / 1e9,
        "pct_mfma_peak": 100 * achieved / PEAK_BF16_TFLOPS,
        "roofline": {"bound": "mfma", "achieved": achieved, "peak": PEAK_BF16_TFLOPS,
                     "unit": "TFLOP/s", "frac": achieved / PEAK_BF16_TFLOPS, "traffic": traffic,
                     "kernel": "attn_fwd_kernel<128,2,64,4,false,1>",
                     "kernel_ms": attn_ms},
    }

    if args.calib_copy_mb > 0:
        src = torch.empty(args.calib_copy_mb << 20, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        src.fill_(1)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        log(f"calibration copy of {args.calib_copy_mb} MiB done")
        del src, dst

    if not args.no_gemm_ref:
        rec["mfma_reference"] = gemm_reference(torch, achieved)
        mr = rec["mfma_reference"]
        log(f"library bf16 GEMM: {mr['random_tflops']:.0f} TF/s on random operands "
            f"({100 * mr['random_frac_of_peak']:.1f}% of peak), {mr['zeros_tflops']:.0f} TF/s on zeros; "
            f"attention kernel at {100 * mr['attention_over_random_gemm']:.1f}% of the random-operand GEMM")

    if not args.no_dense:
        point = run_point(torch, bf1, w, q, k, v, args.warmup, args.reps)
        rec["paper_protocol"] = point
        log(f"two-order protocol: bf1 {point['bf1_ms']:.4f} ms, dense {point.get('dense_ms', 0):.4f} ms,"
            f" speedup {point.get('speedup_vs_dense', 0):.2f}x; PyTorch SDPA {point.get('sdpa_ms', 0):.4f} ms,"
            f" speedup {point.get('speedup_vs_sdpa', 0):.2f}x")

    if not args.no_sweep_device:
        rec["sweep"] = sweep_device(torch, bf1, synth)

    if not args.no_backward:
        bp = backward_point(torch, bf1, synth, w, q, k, v, args.warmup, args.reps)
        rec["backward"] = bp
        log(f"backward: {bp['bwd_ms']:.4f} ms ({bp['bwd_tflops']:.1f} TF/s, {bp['bwd_pct_peak']:.1f}%),"
            f" forward {bp['fwd_ms']:.4f} ms, bwd/fwd {bp['bwd_over_fwd']:.2f}")

    if not args.no_variants:
        vp = variants_point(torch, bf1, w, q, k, v, args.warmup, args.reps)
        rec["route_variants"] = vp
        log("route variants: " + ", ".join(
            f"{kd} {vp[kd]['ms']:.4f} ms (depth {vp[kd]['max_shortest_path']})"
            for kd in ("bf1", "sliding", "static_random")))

    if not args.no_decode:
        rec["decode"] = []
        for name, dw in synth.DECODE_WORKLOADS.items():
            d = decode_point(torch, bf1, synth, dw, args.reps)
            rec["decode"].append(d)
            log(f"decode {name}: step {d['bf1']['step_us_graph']:.1f} us graph / "
                f"{d['bf1']['step_us_eager']:.1f} us eager ({d['bf1']['achieved_GBs']:.0f} GB/s), plan "
                f"{d['bf1']['plan_us_graph']:.1f} us; dense step {d['dense']['step_us_graph']:.1f} us "
                f"({d['dense']['achieved_GBs']:.0f} GB/s); speedup {d['speedup_vs_dense_graph']:.2f}x")

    if not args.no_ttft:
        tt = ttft_point(torch, synth)
        rec["ttft"] = tt
        for n, r in tt["contexts"].items():
            log(f"ttft n={n}: dense {r['dense_ms']:.1f} ms, middle 8 BF1 {r['bf1_middle8_ms']:.1f} ms "
                f"({r['speedup_middle8']:.2f}x), all BF1 {r['bf1_all_ms']:.1f} ms ({r['speedup_all']:.2f}x); "
                f"with PyTorch SDPA as the dense path: {r.get('sdpa_dense_ms', 0):.1f} ms -> "
                f"{r.get('sdpa_bf1_middle8_ms', 0):.1f} ms ({r.get('speedup_middle8_vs_sdpa_dense', 0):.2f}x), "
                f"all BF1 {r.get('speedup_all_vs_sdpa_dense', 0):.2f}x")

    if args.sweep:
        if os.path.dirname(args.sweep_out):
            os.makedirs(os.path.dirname(args.sweep_out), exist_ok=True)
        with open(args.sweep_out, "w") as f:
            for b in (64, 128):
                for sw in synth.sweep(b):
                    sq, sk, sv = synth.make_qkv(sw, device="cuda")
                    r = run_point(torch, bf1, sw, sq, sk, sv, 5, 30)
                    f.write(json.dumps(r) + "\n")
                    f.flush()
                    log(f"sweep n={sw.n} b={b}: bf1 {r['bf1_ms']:.4f} ms ({r['bf1_tflops']:.1f} TF/s,"
                        f" {r['bf1_pct_peak']:.1f}%), dense {r['dense_ms']:.4f} ms"
                        f" ({r['dense_tflops']:.1f} TF/s), speedup {r['speedup_vs_dense']:.2f}x,"
                        f" SDPA {r.get('sdpa_ms', 0):.4f} ms, speedup {r.get('speedup_vs_sdpa', 0):.2f}x")
                    del sq, sk, sv

    if not args.no_cpu_baseline:
        log("cpu baseline (oracle) ...")
        rec["cpu_baseline"] = cpu_baseline(w, args.cpu_seconds, min_seconds=10.0)
        log(f"cpu baseline {rec['cpu_baseline']['value'] * 1e3:.3f} GFLOP/s in "
            f"{rec['cpu_baseline']['seconds']:.1f} s")
        rec["cpu_baseline_configs"] = []
        for name in ("tiny_n512", "qwen_n4096", "qwen_n30001_b2_peaked"):
            cb = cpu_baseline(synth.WORKLOADS[name], 10.0, min_seconds=2.0)
            cb["workload"] = name
            rec["cpu_baseline_configs"].append(cb)
            log(f"cpu baseline {name}: {cb['value'] * 1e3:.3f} GFLOP/s, {cb['gflop']:.2f} GFLOP in "
                f"{cb['seconds']:.1f} s")
    print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    main()
