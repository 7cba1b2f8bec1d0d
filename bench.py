"""Benchmark: one multi-tensor LAMB (or LARS) step per timed iteration.

Default workload: the BERT-Large-shaped parameter set (391 tensors,
335,141,888 fp32 parameters, bf16 gradients), LAMB with the paper's
hyperparameters. Inputs are synthetic, seeded, drawn on the GPU and resident
in HBM before timing starts. Prints ONE JSON line on stdout; diagnostics go
to stderr. Besides the contract's fields the line holds the per-kernel times,
the dominant kernel's roofline, the CPU oracle's rate on a bounded sample,
the latency of single steps timed one by one after the timed region (median,
min, max) and the GPU, runtime and host it ran on.

  python bench.py [--steps K] [--warmup W] [--config 2] [--algo lamb|lars]
                  [--path auto|two-pass] [--chunk ELEMS]
                  [--cpu-seconds S | --no-cpu-baseline]
  python bench.py --copy-probe      # plain copy of known size (counter scale)
  python bench.py --stream-probe    # attainable GB/s of each kernel's access pattern
"""

from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "LAMB step: params updated/sec + achieved HBM GB/s (% peak), BERT-Large fp32"
HBM_PEAK_GBPS = 8000.0  # MI355X HBM3E, published
PROFILES = os.path.join(ROOT, "profiles")
NLAMB_BETA1, NLAMB_EPS = 0.975, 1e-8  # N-LAMB / NN-LAMB settings (Appendix D)
TIMING_EVERY = 4  # kernel-level events on one timed step in four
LATENCY_STEPS = 50  # steps timed one by one after the timed region


def eprint(*a):
    print(*a, file=sys.stderr, flush=True)


def bytes_per_param(algo: str, g_bytes: int, deferred: bool = False):
    """Algorithmic HBM bytes per parameter of (moment pass, apply pass).

    Direct mode: the LAMB moment pass reads x, g, m, v and writes m, v; the
    apply pass reads x, m, v and writes x (N-LAMB and NN-LAMB also read g
    there). LARS reads x, g, m and writes m, then reads x, m and writes x.
    Deferred mode (skip on a non-finite gradient): the moment pass only
    reads; the apply pass reads x, g and the old moments and writes x and the
    new moments.
    """
    state = 8 if algo != "lars" else 4          # m, v  /  m
    moment_reads = 4 + g_bytes + state
    if deferred:
        return moment_reads, moment_reads + 4 + state
    needs_g = algo in ("nlamb", "nnlamb")
    return moment_reads + state, 4 + state + 4 + (g_bytes if needs_g else 0)


def avg_one_ms(total_ms: float, recorded: int) -> float:
    return total_ms / recorded if recorded else 0.0


def single_pass_bytes(algo: str, g_bytes: int) -> int:
    """Algorithmic HBM bytes per parameter of the single-pass kernel: x, g and
    the moments read once, the moments and x written once."""
    state = 8 if algo != "lars" else 4
    return 4 + g_bytes + state + state + 4


def algo_label(algo: str) -> str:
    return {"lamb": "LAMB", "lars": "LARS", "nlamb": "N-LAMB", "nnlamb": "NN-LAMB"}[algo]


def _strip_comments(src: str) -> str:
    """C/C++ source without // and /* */ comments, blank lines and trailing
    blanks (the sources hashed here hold no string literal with either
    comment sequence)."""
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    src = re.sub(r"//[^\n]*", "", src)
    return "\n".join(line.rstrip() for line in src.splitlines() if line.strip())


def kernel_source_hash() -> str:
    """Hash of what the kernels' machine code depends on: the kernel source,
    the layout header it shares with the host side (both without comments),
    and the compile flags."""
    from paper_1904_00962_amd import build as hb
    h = hashlib.sha256()
    for p in (os.path.join(hb.CSRC, "lamb_kernels.hip"), os.path.join(hb.CSRC, "lamb_internal.h")):
        with open(p) as f:
            h.update(_strip_comments(f.read()).encode())
    h.update(" ".join(hb.HIPCC_FLAGS).encode())
    return h.hexdigest()[:16]


def counter_traffic(kernel: str, workload: str, src_hash: str):
    """HBM bytes per launch of `kernel` ("moments" or "single_pass") from the
    committed rocprofv3 counter summary for this workload, or None if absent
    or stale."""
    path = os.path.join(PROFILES, "lamb_%s_%s_traffic.md" % (kernel, workload))
    if not os.path.exists(path):
        return None
    text = open(path).read()
    m = re.search(r"kernel_source_hash:\s*(\w+)", text)
    t = re.search(r"hbm_bytes_per_launch:\s*([0-9.eE+]+)", text)
    if not m or not t or m.group(1) != src_hash:
        return None
    return float(t.group(1))


def copy_probe(args) -> None:
    """A plain device-to-device copy of known size: FETCH_SIZE / WRITE_SIZE of
    this kernel calibrate the counters (bytes per counted KiB)."""
    import torch
    n = args.copy_elems
    src = torch.ones(n, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record()
    for _ in range(args.steps):
        dst.copy_(src)
    end.record()
    torch.cuda.synchronize()
    ms = start.elapsed_time(end) / args.steps
    print(json.dumps({"probe": "copy", "bytes_read": 4 * n, "bytes_written": 4 * n,
                      "ms": ms, "GBps": 8 * n / ms / 1e6}), flush=True)


PATTERNS = {"single_pass": 0, "moments": 1, "apply": 2, "read": 3, "copy": 4}


def pattern_bytes(pattern: str, g_bytes: int) -> int:
    """Bytes per element of a stream pattern (include/stream_probe.h)."""
    return {"single_pass": 4 + g_bytes + 8 + 12, "moments": 4 + g_bytes + 8 + 8,
            "apply": 12 + 4, "read": 12 + g_bytes, "copy": 8}[pattern]


BEST_STREAM_TILES = (256, 512, 1024, 2048)


def stream_rate(pattern: str, n: int, g_bf16: bool, tile: int, layer_tiles: int = 0,
                reps: int = 20) -> float:
    """Attainable GB/s of a stream with `pattern`'s access pattern over n
    elements (the stream probe library), timed with events on torch's current
    stream, on buffers of its own."""
    import ctypes

    import torch

    from paper_1904_00962_amd import build as hb
    if not os.path.exists(hb.PROBE_LIBRARY):
        raise RuntimeError("stream probe library %s is missing; run the build" % hb.PROBE_LIBRARY)
    lib = ctypes.CDLL(hb.PROBE_LIBRARY)
    lib.stream_probe.argtypes = [ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p,
                                 ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int32,
                                 ctypes.c_int64, ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p]
    x, m, v = (torch.zeros(n, dtype=torch.float32, device="cuda") for _ in range(3))
    g = torch.zeros(n, dtype=torch.bfloat16 if g_bf16 else torch.float32, device="cuda")
    stream = torch.cuda.current_stream().cuda_stream

    def run():
        rc = lib.stream_probe(PATTERNS[pattern], x.data_ptr(), m.data_ptr(), v.data_ptr(),
                              g.data_ptr(), int(g_bf16), n, tile, layer_tiles, stream)
        if rc != 0:
            raise RuntimeError("stream_probe failed with %d" % rc)

    for _ in range(3):
        run()
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(reps):
        run()
    b.record()
    torch.cuda.synchronize()
    ms = a.elapsed_time(b) / reps
    rate = pattern_bytes(pattern, 2 if g_bf16 else 4) * n / ms / 1e6
    del x, m, v, g
    torch.cuda.empty_cache()
    return rate


def stream_probe_all() -> None:
    """Every pattern over the BERT-Large parameter count, one JSON line."""
    out = {"probe": "stream", "elements": 335141888, "g": "bf16"}
    from paper_1904_00962_amd import _lib
    chunk = int(_lib.lamb_chunk_table([1 << 20], 0)[2][0])  # a plan's default chunk
    for pattern, tile in (("single_pass", 8192), ("moments", chunk), ("apply", chunk),
                          ("read", 2048), ("copy", 512)):
        out[pattern + "_GBps"] = stream_rate(pattern, 335141888, True, tile)
    # the single pass's own layout: 1024-element blocks dealt over layers of 512 tiles
    out["single_pass_dealt_GBps"] = stream_rate("single_pass", 335141888, True, 8192, 512)
    for tile in BEST_STREAM_TILES:
        out["single_pass_tile%d_GBps" % tile] = stream_rate("single_pass", 335141888, True, tile)
    print(json.dumps(out), flush=True)


def step_latencies(opt, n: int) -> dict:
    """Latency of single steps: an event pair on the step's stream around
    each of ``n`` more steps, after the timed region (the events add a little
    to each step, so the timed region keeps the throughput figure)."""
    import torch
    stream = torch.cuda.current_stream()
    pairs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
             for _ in range(n)]
    torch.cuda.synchronize()
    for a, b in pairs:
        a.record(stream)
        opt.step()
        b.record(stream)
    torch.cuda.synchronize()
    ms = sorted(a.elapsed_time(b) for a, b in pairs)
    mid = len(ms) // 2
    median = ms[mid] if len(ms) % 2 else 0.5 * (ms[mid - 1] + ms[mid])
    return {"median_ms": median, "min_ms": ms[0], "max_ms": ms[-1], "steps": n}


def environment() -> dict:
    """The GPU, runtime and host the line was measured on."""
    import torch
    props = torch.cuda.get_device_properties(0)
    host = ""
    try:
        with open("/proc/cpuinfo") as f:
            for ln in f:
                if ln.startswith("model name"):
                    host = ln.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return {"gpu": props.name, "arch": getattr(props, "gcnArchName", ""),
            "compute_units": props.multi_processor_count, "hip": torch.version.hip,
            "torch": torch.__version__, "host_cpu": host}


def cpu_sample(ps, xs, grads):
    """Host copies of the leading tensors covering at least a third of the
    parameters: the bounded sample the oracle is timed on."""
    import numpy as np

    from paper_1904_00962_amd import paramsets

    idx, total = [], 0
    for i, spec in enumerate(ps.tensors):
        idx.append(i)
        total += spec.numel
        if total >= ps.numel // 3:
            break
    hx = [paramsets.host_array(xs[i]).copy() for i in idx]
    hg = [paramsets.host_array(grads[i]).copy() for i in idx]
    hm = [np.zeros_like(h) for h in hx]
    hv = [np.zeros_like(h) for h in hx]
    return idx, total, hx, hg, hm, hv


def cpu_baseline(ps, sample, algo, budget_s: float):
    """Time the oracle (single-threaded C, as it stands) on the sample: whole
    steps over it until ``budget_s`` seconds have been spent (at least one,
    at most 100)."""
    import numpy as np

    import oracle

    idx, total, hx, hg, hm, hv = sample
    o = oracle.load()
    wd = [ps.wd_mask()[i] for i in idx]
    f = lambda a: float(np.float32(a))  # noqa: E731
    done, spent = 0, 0.0
    while done == 0 or (spent < budget_s and done < 100):
        t0 = time.perf_counter()
        if algo == "lamb":
            o.lamb_step(hx, hg, hm, hv, wd, lr=f(ps.lr), beta1=f(ps.beta1), beta2=f(ps.beta2),
                        eps=f(ps.eps), weight_decay=f(ps.weight_decay), gamma_l=f(ps.gamma_l),
                        gamma_u=f(ps.gamma_u), step=done + 1)
        elif algo in ("nlamb", "nnlamb"):
            o.nlamb_step(hx, hg, hm, hv, wd, lr=f(ps.lr), beta1=f(NLAMB_BETA1), beta2=f(ps.beta2),
                         eps=f(NLAMB_EPS), weight_decay=f(ps.weight_decay),
                         gamma_l=f(ps.gamma_l), gamma_u=f(ps.gamma_u), step=done + 1,
                         nesterov_v=algo == "nnlamb")
        else:
            o.lars_step(hx, hg, hm, wd, lr=f(ps.lars_lr), momentum=f(ps.lars_momentum),
                        weight_decay=f(ps.weight_decay), gamma_l=f(ps.gamma_l),
                        gamma_u=f(ps.gamma_u), trust_coef=f(ps.lars_trust_coef))
        spent += time.perf_counter() - t0
        done += 1
    return {"value": total * done / spent, "unit": "params/s", "cores": 1, "kind": "oracle",
            "sample": "%d %s step(s) over the first %d of %d tensors (%d of %d params), "
                      "single-threaded C oracle, %.1f s" % (done, algo.upper(), len(idx),
                                                            ps.n_tensors, total, ps.numel, spent),
            "host_cpus": os.cpu_count()}


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawTextHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--config", type=int, default=2)
    ap.add_argument("--algo", choices=("lamb", "lars", "nlamb", "nnlamb"), default="lamb")
    ap.add_argument("--chunk", type=int, default=0, help="elements per chunk (0 = default)")
    ap.add_argument("--path", choices=("auto", "two-pass"), default="auto",
                    help="auto: the single-pass kernel for every layer that fits one round of tiles and for the last tiles of larger ones")
    ap.add_argument("--norm", choices=("l2", "l1", "linf"), default="l2",
                    help="layer norm (Appendix F)")
    ap.add_argument("--grad-scale", type=float, default=1.0)
    ap.add_argument("--skip-nonfinite", action="store_true",
                    help="deferred-write mode that skips steps with NaN/Inf gradients")
    ap.add_argument("--bf16-copy", action="store_true",
                    help="the apply pass also writes a bf16 copy of x")
    ap.add_argument("--shard", type=int, default=1,
                    help="time one rank's share of a step sharded N ways: the first 1/N slice "
                         "of every tensor (the kernels at that rank's real shape)")
    ap.add_argument("--cpu-seconds", type=float, default=10.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-probe", action="store_true")
    ap.add_argument("--stream-probe", action="store_true",
                    help="attainable GB/s of each kernel's access pattern, then exit")
    ap.add_argument("--copy-elems", type=int, default=1 << 28)
    args = ap.parse_args()

    if args.gpus != 1:
        print("bench.py measures one GPU: the optimizer step runs on a single MI355X; "
              "--gpus %d is not supported" % args.gpus, file=sys.stderr)
        return 2

    import torch
    if not torch.cuda.is_available():
        eprint("bench.py needs a GPU")
        return 1
    if args.copy_probe:
        copy_probe(args)
        return 0
    if args.stream_probe:
        stream_probe_all()
        return 0

    from paper_1904_00962_amd import _lib, paramsets
    from paper_1904_00962_amd.optim import LAMB, LARS

    _lib.load()  # fail loudly before any work if the HIP library is missing
    ps = paramsets.get(args.config)
    eprint("drawing %s: %d tensors, %d params (g %s)" % (ps.name, ps.n_tensors, ps.numel,
                                                          ps.g_dtype))
    xs = paramsets.draw_params(ps, device="cuda")
    grads = paramsets.draw_grads(ps, 1, device="cuda")
    if args.shard > 1:
        # rank 0's slice of each tensor's flat range: ceil(n / N) rounded up
        # to a multiple of 4 elements, so every rank's slice starts 16-byte aligned
        def share(n):
            per_rank = -(-n // args.shard)          # ceil(n / N)
            return min(n, (per_rank + 3) // 4 * 4)
        lens = [share(x.numel()) for x in xs]
        xs = [x[:k] for x, k in zip(xs, lens)]
        grads = [g[:k] for g, k in zip(grads, lens)]
    # the plan's fault word is read after the timed region (opt.check()), not
    # inside it
    extra = dict(norm=args.norm, grad_scale=args.grad_scale, skip_nonfinite=args.skip_nonfinite,
                 wd_mask=ps.wd_mask(), chunk_elems=args.chunk, path=args.path, check_every=0)
    if args.algo == "lamb":
        opt = LAMB(xs, grads, lr=ps.lr, betas=(ps.beta1, ps.beta2), eps=ps.eps,
                   weight_decay=ps.weight_decay, clamp=(ps.gamma_l, ps.gamma_u), **extra)
    elif args.algo in ("nlamb", "nnlamb"):
        opt = LAMB(xs, grads, lr=ps.lr, betas=(NLAMB_BETA1, ps.beta2), eps=NLAMB_EPS,
                   weight_decay=ps.weight_decay, clamp=(ps.gamma_l, ps.gamma_u),
                   variant="n-lamb" if args.algo == "nlamb" else "nn-lamb", **extra)
    else:
        opt = LARS(xs, grads, lr=ps.lars_lr, momentum=ps.lars_momentum,
                   weight_decay=ps.weight_decay, clamp=(ps.gamma_l, ps.gamma_u),
                   trust_coef=ps.lars_trust_coef, **extra)
    if args.bf16_copy:
        opt.attach_bf16_copies("allocate")
    n_tensors, n_chunks, chunk = _lib.lamb_plan_info(opt.plan)
    tiles_per_tensor, n_tiles, tile_groups, single_elems = _lib.lamb_plan_tiles(opt.plan, True)
    single = args.path == "auto"
    P = sum(x.numel() for x in xs)
    # elements on the single pass: whole layers, and the tails of layers
    # larger than one round (their heads take the two-pass kernels)
    P_single = sum(single_elems) if single else 0
    checked = single and args.skip_nonfinite and P_single > 0

    # The oracle's sample is copied out before the GPU steps move x; the
    # oracle itself runs after the GPU timing, so the GPU is not left idle
    # (and clocked down) right before the timed steps.
    sample = None if args.no_cpu_baseline else cpu_sample(ps, xs, grads)

    for _ in range(args.warmup):
        opt.step()
    torch.cuda.synchronize()
    # HIP events around the kernels of every TIMING_EVERY-th timed step
    _lib.lamb_plan_set_timing(opt.plan, args.steps, TIMING_EVERY)
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record()
    for _ in range(args.steps):
        opt.step()
    end.record()
    torch.cuda.synchronize()
    total_ms = start.elapsed_time(end)
    (k_mom, k_fin, k_app, k_one, k_chk), recorded = _lib.lamb_plan_timing(opt.plan)
    _lib.lamb_plan_set_timing(opt.plan, 0)
    opt.check()
    ratios = opt.ratios.cpu()
    if not torch.isfinite(ratios).all():
        eprint("non-finite trust ratio after the timed steps")
        return 1
    latency = step_latencies(opt, LATENCY_STEPS)
    opt.check()
    eprint("single-step latency over %d steps: median %.4f ms, min %.4f ms, max %.4f ms"
           % (latency["steps"], latency["median_ms"], latency["min_ms"], latency["max_ms"]))
    # What a plain stream of the dominant kernel's traffic reaches: the same
    # reads and writes over the same parameters, no arithmetic. `attainable`
    # is the fastest of contiguous tiles of 256 to 2048 elements per
    # workgroup; `same_layout` keeps the kernel's own elements per workgroup
    # (and, for the single pass, its dealt block layout).
    dom_is_single = avg_one_ms(k_one, recorded) >= avg_one_ms(k_mom, recorded)
    dom_pattern = "single_pass" if dom_is_single else "moments"
    dom_elems = P_single if dom_is_single else P - P_single
    same_layout = best_stream = None
    if not args.skip_nonfinite and not args.bf16_copy and args.algo != "lars" and dom_elems:
        # the single pass deals its layers' blocks over their tiles; its largest
        # layers on BERT-Large have 512 tiles
        same_layout = stream_rate(dom_pattern, dom_elems, ps.g_dtype == "bf16",
                                  1024 * tile_groups if dom_is_single else chunk,
                                  512 if dom_is_single else 0)
        eprint("stream probe (%s pattern, %d elements, the kernel's layout): %.0f GB/s"
               % (dom_pattern, dom_elems, same_layout))
        best_stream = max((stream_rate(dom_pattern, dom_elems, ps.g_dtype == "bf16", t), t)
                          for t in BEST_STREAM_TILES)
        eprint("best plain stream of that traffic: %.0f GB/s (%d elements per workgroup)"
               % best_stream)
    cpu = None
    if sample is not None:
        eprint("timing the CPU oracle (budget %.0f s)" % args.cpu_seconds)
        cpu = cpu_baseline(ps, sample, args.algo, args.cpu_seconds)
        eprint("cpu baseline: %.3e params/s (%s)" % (cpu["value"], cpu["sample"]))

    ms_step = total_ms / args.steps
    P_rest = P - P_single
    g_bytes = 2 if ps.g_dtype == "bf16" else 4
    copy_bytes = 2 if args.bf16_copy else 0  # the bf16 working copy of x
    # a checked skip step runs the direct kernels after a read-only check of g
    b_mom, b_app = bytes_per_param(args.algo, g_bytes, args.skip_nonfinite and not checked)
    b_app += copy_bytes
    b_one = single_pass_bytes(args.algo, g_bytes) + copy_bytes
    b_chk = g_bytes if checked else 0
    avg_mom, avg_fin, avg_app, avg_one, avg_chk = (k / recorded for k in
                                                   (k_mom, k_fin, k_app, k_one, k_chk))
    gbps = lambda b, n, ms: b * n / ms / 1e6 if ms > 0 and n else 0.0  # noqa: E731
    mom_gbps = gbps(b_mom, P_rest, avg_mom)
    app_gbps = gbps(b_app, P_rest, avg_app)
    one_gbps = gbps(b_one, P_single, avg_one)
    step_bytes = b_one * P_single + (b_mom + b_app) * P_rest + b_chk * P
    step_gbps = step_bytes / ms_step / 1e6
    workload = ps.name if args.shard == 1 else "%s-shard-1of%d" % (ps.name, args.shard)
    src_hash = kernel_source_hash()
    default_mode = (args.algo == "lamb" and args.norm == "l2" and not args.skip_nonfinite
                    and not args.bf16_copy)
    algo_name = algo_label(args.algo)
    g_name = "bf16" if g_bytes == 2 else "f32"
    # the roofline entry covers the kernel that takes the most time
    if avg_one >= avg_mom:
        dom = dict(kernel="fused_kernel<%s, %s, %s, %d groups>" % (algo_name, g_name, args.norm,
                                                                  tile_groups),
                   achieved=one_gbps, bytes_per_launch=b_one * P_single,
                   traffic=counter_traffic("single_pass", workload, src_hash)
                   if default_mode else None)
    else:
        dom = dict(kernel="moments_kernel<%s, %s, %s%s>" % (
                       algo_name, g_name, args.norm, ", deferred" if args.skip_nonfinite else ""),
                   achieved=mom_gbps, bytes_per_launch=b_mom * P_rest,
                   traffic=counter_traffic("moments", workload, src_hash)
                   if default_mode else None)
    eprint("step %.4f ms | check %.4f ms | single pass %.4f ms (%.0f GB/s, %d params) | moments "
           "%.4f ms (%.0f GB/s) | finalize %.4f ms | apply %.4f ms (%.0f GB/s, %d params) | whole "
           "step %.0f GB/s" % (ms_step, avg_chk, avg_one, one_gbps, P_single, avg_mom, mom_gbps,
                               avg_fin, avg_app, app_gbps, P_rest, step_gbps))
    line = {
        "metric": METRIC,
        "value": P / (ms_step / 1e3),
        "unit": "params/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {
            "workload": "%s %s step: %d tensors, %d fp32 params, %s gradients"
                        % (workload, algo_name, n_tensors, P, ps.g_dtype),
            "algo": args.algo, "tensors": n_tensors, "params": P, "grad_dtype": ps.g_dtype,
            "path": args.path, "single_pass_params": P_single, "single_pass_tiles": n_tiles,
            "tile_elems": 1024 * tile_groups if single else 0,
            "chunk_elems": chunk, "chunks": n_chunks, "norm": args.norm,
            "grad_scale": args.grad_scale, "skip_nonfinite": args.skip_nonfinite,
            "bf16_copy": args.bf16_copy,
            "shard": args.shard, "seed_x": 1000 * ps.cfg,
            "seed_g": 1000 * ps.cfg + 1,
        },
        "hbm_GBps": step_gbps,
        "hbm_frac_of_peak": step_gbps / HBM_PEAK_GBPS,
        "bytes_per_param": step_bytes / P,
        "kernels_ms": {"single_pass": avg_one, "moments": avg_mom, "finalize": avg_fin,
                       "apply": avg_app, "finite_check": avg_chk, "steps_sampled": recorded},
        "roofline": {
            "bound": "hbm", "kernel": dom["kernel"], "achieved": dom["achieved"],
            "peak": HBM_PEAK_GBPS, "unit": "GB/s", "frac": dom["achieved"] / HBM_PEAK_GBPS,
            "traffic": dom["traffic"], "bytes_per_launch": dom["bytes_per_launch"],
            "kernel_source_hash": src_hash,
            "attainable": None if best_stream is None else {
                "GBps": best_stream[0], "frac": dom["achieved"] / best_stream[0],
                "how": "fastest plain stream of the kernel's reads and writes over the same "
                       "parameters, no arithmetic (libstream_probe): contiguous tiles of %d "
                       "elements per workgroup, the best of %s"
                       % (best_stream[1], list(BEST_STREAM_TILES)),
                "same_layout_GBps": same_layout,
                "same_layout_how": "the same stream with the kernel's own elements per "
                                   "workgroup and block layout"},
        },
        "cpu_baseline": cpu,
        "latency": latency,
        "env": environment(),
    }
    if cpu:
        cpu["gpu_speedup"] = line["value"] / cpu["value"]
    print(json.dumps(line), flush=True)
    opt.close()
    return 0


if __name__ == "__main__":
    sys.exit(main())
