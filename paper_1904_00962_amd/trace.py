"""Per-tile timeline of the single-pass kernel (lamb_plan_set_trace).

    python -m paper_1904_00962_amd.trace [--config 2] [--algo lamb|lars] [--steps 3]

Runs warm-up steps of a parameter set's step (synthetic inputs, as bench.py),
then traced steps, and prints a Markdown summary of the last one: each tile's
read phase (start to partial norms done), wait (to its layer's step scale)
and write phase; how far apart the tiles of a round finish reading; the
microseconds in which the streaming demand (each tile's reads spread over its
read phase, its x writes over its write phase) stays below given rates; and
how the read phase depends on the order in which workgroups were dispatched
onto their CUs and on their XCD. Measurement only.
"""

from __future__ import annotations

import argparse
import sys

import numpy as np

TICK_US = 0.01  # the trace clock runs at 100 MHz


def run(cfg: int, algo: str, steps: int, warmup: int):
    import torch

    from . import _lib, paramsets
    from .optim import LAMB, LARS

    ps = paramsets.get(cfg)
    xs = paramsets.draw_params(ps, device="cuda")
    gs = paramsets.draw_grads(ps, 1, device="cuda")
    if algo == "lars":
        opt = LARS(xs, gs, lr=ps.lars_lr, momentum=ps.lars_momentum, weight_decay=ps.weight_decay,
                   clamp=(ps.gamma_l, ps.gamma_u), trust_coef=ps.lars_trust_coef,
                   wd_mask=ps.wd_mask(), check_every=0)
    else:
        opt = LAMB(xs, gs, lr=ps.lr, betas=(ps.beta1, ps.beta2), eps=ps.eps,
                   weight_decay=ps.weight_decay, clamp=(ps.gamma_l, ps.gamma_u),
                   wd_mask=ps.wd_mask(), check_every=0)
    per, n_tiles, groups, elems = _lib.lamb_plan_tiles(opt.plan, True)
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    # the plan's schedule over the elements each layer has on the single pass
    et, _, el, _, tiles, width, _ = _lib.lamb_tile_schedule(elems, 4 * cus, groups)
    assert len(et) == n_tiles and list(tiles) == list(per)
    for _ in range(warmup):
        opt.step()
    trace = torch.zeros(4 * n_tiles, dtype=torch.int64, device="cuda")
    ms = []
    for _ in range(steps):
        trace.zero_()
        _lib.lamb_plan_set_trace(opt.plan, trace.data_ptr())
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        opt.step()
        b.record()
        torch.cuda.synchronize()
        _lib.lamb_plan_set_trace(opt.plan, 0)
        ms.append(a.elapsed_time(b))
    opt.check()
    stamps = trace.cpu().numpy().reshape(-1, 4)
    info = dict(name=ps.name, algo=algo, tensors=ps.n_tensors, params=ps.numel,
                g_dtype=ps.g_dtype, groups=groups, width=width, step_ms=ms,
                bytes_per_param=(18 if algo == "lars" else 26) + (2 if ps.g_dtype == "f32" else 0))
    opt.close()
    return stamps, np.asarray(et), np.asarray(el), np.asarray(tiles), info


def summarize(stamps, et, el, tiles, info) -> str:
    valid = et >= 0
    idx = np.nonzero(valid)[0]
    t = stamps[valid].astype(np.float64) * TICK_US
    t -= t[:, 0].min()
    read, wait, write = t[:, 1] - t[:, 0], t[:, 2] - t[:, 1], t[:, 3] - t[:, 2]
    span = t[:, 3].max()
    elems = el[valid].astype(np.float64)
    team = tiles[et[valid]]
    width = int(info["width"])
    rnd = idx // width
    bpp = info["bytes_per_param"]
    out = ["Workload: %s %s step, %d tensors, %d params (%s gradients); tiles of %d elements, "
           "rounds of %d tiles." % (info["name"], info["algo"].upper(), info["tensors"],
                                    info["params"], info["g_dtype"], 1024 * info["groups"], width),
           "Traced steps: %s ms (the last is summarized)." % ", ".join("%.4f" % v
                                                                   for v in info["step_ms"]),
           "", "Single-pass kernel span %.1f us for %d tiles in %d rounds: %.0f GB/s at %d B/param."
           % (span, len(t), rnd.max() + 1, elems.sum() * bpp / span / 1e3, bpp), "",
           "| phase | mean us | p50 | p90 | max |", "|---|---|---|---|---|"]
    for name, v in (("read (start to partial norms)", read), ("wait (to the layer's scale)", wait),
                    ("write (x issued)", write)):
        out.append("| %s | %.2f | %.2f | %.2f | %.2f |" % (name, v.mean(), np.median(v),
                                                         np.percentile(v, 90), v.max()))
    spread = [t[rnd == r, 1].max() - t[rnd == r, 1].min() for r in range(rnd.max() + 1)]
    late = [t[rnd == r, 2].max() - t[rnd == r, 1].max() for r in range(rnd.max() + 1)]
    out += ["", "Per round: the tiles finish reading %.1f us apart (median over rounds; max %.1f), "
            "and the last scale is known %.1f us after the last read ends (median)."
            % (np.median(spread), max(spread), np.median(late)),
            "Kernel tail after the last read ends: %.1f us." % (span - t[:, 1].max())]
    # streaming demand: reads over the read phase, x writes over the write phase
    nb = int(span) + 2
    demand = np.zeros(nb)
    for s0, s1, nbytes in ((t[:, 0], t[:, 1], (bpp - 4) * elems), (t[:, 2], t[:, 3], 4 * elems)):
        for a, b, q in zip(s0, np.maximum(s1, s0 + 0.01), nbytes):
            ia, ib = int(a), int(b)
            rate = q / (b - a)
            for i in range(ia, ib + 1):
                lo, hi = max(a, i), min(b, i + 1)
                if hi > lo:
                    demand[i] += rate * (hi - lo)
    gbps = demand[: int(span)] / 1e3
    out += ["", "Microseconds of the span in which the streaming demand stays below a rate:", "",
            "| below | us | share of span |", "|---|---|---|"]
    for thr in (2000, 4000, 5000, 6000):
        n = int((gbps < thr).sum())
        out.append("| %d GB/s | %d | %.1f%% |" % (thr, n, 100.0 * n / max(1, int(span))))
    # systematic effects on the read phase of multi-tile layers, normalized per round
    norm = read.copy()
    for r in np.unique(rnd):
        m = rnd == r
        norm[m] = read[m] / read[m].mean()
    multi = team > 1
    w = idx % width

    def rel(mask):
        return "%.3f" % norm[mask].mean() if mask.any() else "-"

    slot = w * 4 // width
    out += ["", "Read phase of tiles of multi-tile layers, relative to their round's mean:", "",
            "| by | groups |", "|---|---|",
            "| dispatch order on the CU (workgroup index * 4 / round) | %s |"
            % ", ".join("%d: %s" % (k, rel(multi & (slot == k))) for k in range(4)),
            "| XCD (workgroup index mod 8) | %s |"
            % ", ".join("%d: %s" % (k, rel(multi & (w % 8 == k))) for k in range(8))]
    grid = np.full((width, rnd.max() + 1), np.nan)
    grid[w[multi], rnd[multi]] = norm[multi]
    a, b = grid[:, :-1].ravel(), grid[:, 1:].ravel()
    ok = ~np.isnan(a) & ~np.isnan(b)
    if ok.sum() > 2:
        out.append("")
        out.append("A workgroup's relative read time in one round and the next correlate %.2f."
                   % np.corrcoef(a[ok], b[ok])[0, 1])
    return "\n".join(out)


def main(argv=None) -> int:
    ap = argparse.ArgumentParser(description=__doc__,
                                 formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--config", type=int, default=2)
    ap.add_argument("--algo", choices=("lamb", "lars"), default="lamb")
    ap.add_argument("--steps", type=int, default=3)
    ap.add_argument("--warmup", type=int, default=20)
    args = ap.parse_args(argv)
    stamps, et, el, tiles, info = run(args.config, args.algo, args.steps, args.warmup)
    print(summarize(stamps, et, el, tiles, info), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
