"""Throughput of the AVQ-Attention forward pass on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W]
    python bench.py --sweep [--steps K] [--warmup W]
    python bench.py --codebook-update [--steps K] [--warmup W]

Before the W warm-up steps, whole untimed steps run for --warmup-ms of wall
time (at least 10; reported as "preheat"): from idle the GPU clock takes some
tens of milliseconds to come up, and steps timed before that measure the ramp.

One step is the whole forward pass over one batch of synthetic inputs
already resident in HBM: avq_assign_aggregate (the precompute of Alg. 1) ->
avq_attention_fwd (--unfused-precompute: avq_assign -> avq_aggregate for the
first).
The workload is the N = 16384 one (B=2, H=16, d=128, M0=256 parents with 8
children each, P=32, query block 128, bf16). Prints one JSON line:

* value: query-token*heads per second of the whole step, B*H*N / t_step;
* roofline: the fused attention kernel (the dominant one) against the bf16
  MFMA peak, its algorithmic flops 4 d (M0 + P Ch) per query-head divided by
  its average launch duration over the timed steps (HIP events on the launch
  stream after each entry point, the end of one being the start of the next);
  traffic is the
  HBM bytes per launch from the committed rocprofv3 counter summary, or null
  if the kernel source changed since those counters were taken;
* cpu_baseline: the fp64 oracle timed on the host cores, whole passes over
  the same workload repeated for at least --cpu-seconds.

--sweep runs the sequence-length sweep of the scaling analysis instead
(Sec. 5: B=4, H=12, d=64, N from 1k to 64k, flat and tree codebooks): one
JSON line per workload with the median step time and the per-kernel medians,
then one line with the fitted log-log slopes of step time against N and
against the effective codebook size (linear scaling is slope 1).
"""
from __future__ import annotations

import argparse
import dataclasses
import hashlib
import json
import math
import os
import re
import sys
import time
from pathlib import Path

ROOT = Path(__file__).resolve().parent
sys.path.insert(0, str(ROOT))

METRIC = "AVQ attention fwd query-tokens·heads/sec at N=16384; % bf16 MFMA peak"
UNIT = "query-token*heads/s"
PEAK_BF16_TFLOPS = 2500.0  # MI355X dense bf16 MFMA
PEAK_F32_TFLOPS = 157.3     # MI355X dense fp32 MFMA
KERNEL_SRC = ROOT / "paper_2607_12789_amd" / "csrc" / "avq_attention.hip"
TRAFFIC_SUMMARY = ROOT / "profiles" / "attention_fwd_c4_traffic.md"


def kernel_hash() -> str:
    """The attention kernel's sources and the compiler flags they are built with."""
    from paper_2607_12789_amd.build import COMPILE_FLAGS
    h = hashlib.sha256()
    for name in ("avq_attention.hip", "avq_common.hpp", "avq_packed.hpp"):
        h.update((KERNEL_SRC.parent / name).read_bytes())
    h.update(" ".join(COMPILE_FLAGS).encode())
    return h.hexdigest()[:16]


def read_traffic():
    """HBM bytes per launch of the attention kernel from the committed counter
    summary, if it was taken on the current kernel source."""
    if not TRAFFIC_SUMMARY.exists():
        return None
    text = TRAFFIC_SUMMARY.read_text()
    m_hash = re.search(r"kernel source hash:\s*`?([0-9a-f]+)`?", text)
    m_bytes = re.search(r"HBM bytes per launch:\s*([0-9.eE+]+)", text)
    if not m_hash or not m_bytes or m_hash.group(1) != kernel_hash():
        return None
    return float(m_bytes.group(1))


def cpu_baseline(x, w, min_seconds: float, max_passes: int):
    """The oracle, as it is, on the host cores: whole forward passes over the
    full workload, repeated until min_seconds of wall time have been spent."""
    import oracle
    passes = 0
    t0 = time.perf_counter()
    while True:
        oracle.forward(x["Q"], x["K"], x["V"], x["Cp"], x["Cc"], w.P, w.block_q)
        passes += 1
        dt = time.perf_counter() - t0
        if dt >= min_seconds or passes >= max_passes:
            break
    qh = w.B * w.H * w.N
    return {"value": passes * qh / dt, "unit": UNIT, "cores": oracle.num_threads(),
            "kind": "oracle",
            "sample": f"{passes} whole forward passes of the same workload ({qh} query-heads "
                      f"each, assign + aggregate + attention in fp64) in {dt:.1f} s wall"}


class Runner:
    """Device buffers of one workload and its timed step (the three entry
    points on torch's current stream)."""

    def __init__(self, w, x, dev, tiled=False, order=None, fused=True):
        import torch
        from paper_2607_12789_amd import avq
        self.avq, self.w, self.tiled, self.fused = avq, w, tiled, fused
        self.order = None if order is None else order.to(dev)
        self.xd = {k: v.to(dev) for k, v in x.items()}
        B, H, N, d = w.B, w.H, w.N, w.d
        self.par = torch.empty((B, H, N), dtype=torch.int32, device=dev)
        self.code = torch.empty_like(self.par)
        self.packed = torch.empty((B, H, avq.packed_bytes(w.torch_dtype, w.M0, w.Ch, d)),
                                  dtype=torch.uint8, device=dev)
        self.counts = torch.empty((B, H, w.Mtot), dtype=torch.int32, device=dev)
        self.Y = torch.empty_like(self.xd["Q"])
        # the step's entry points in order, each timed by the events around it
        self.stages = (["assign_aggregate"] if fused else ["assign", "aggregate"]) + \
            ["attention_fwd"]

    def step(self, ev=None):
        # ev: one event recorded after each entry point (HIP events on the
        # stream the kernels are launched on, which is torch's current one)
        avq, w, xd = self.avq, self.w, self.xd
        if self.fused:
            avq.assign_aggregate(xd["K"], xd["V"], xd["Cp"], xd["Cc"], self.par, self.code,
                                 self.packed, self.counts)
        else:
            avq.assign(xd["K"], xd["Cp"], xd["Cc"], self.par, self.code)
            if ev: ev[0].record()
            avq.aggregate(xd["V"], self.code, w.M0, w.Ch, self.packed, self.counts)
        if ev: ev[-2].record()
        avq.attention_fwd(xd["Q"], xd["Cp"], xd["Cc"], self.packed, w.P, w.block_q, Y=self.Y,
                          tiled_importance=self.tiled, query_order=self.order)
        if ev: ev[-1].record()

    def timed(self, steps: int, warmup: int, cold: bool = False, warmup_ms: float = 200.0):
        """Runs the pre-heat (steps for warmup_ms of wall time), warmup
        untimed steps, and then steps timed steps; returns (wall ms per step,
        per-step event durations [steps][len(stages)] in ms, pre-heat steps
        run). Each entry point is timed from the event before it (the
        previous entry point's, or the start event) to its own. cold: a 1 GiB
        fill before each step, with its own start event after the fill,
        evicts the caches."""
        import torch
        flush = torch.empty(1 << 28, dtype=torch.float32, device=self.Y.device) if cold else None
        preheat = warm_up(self.step, warmup, warmup_ms)
        n = len(self.stages)
        evs = [[torch.cuda.Event(enable_timing=True) for _ in range(n)] for _ in range(steps)]
        starts = [torch.cuda.Event(enable_timing=True) for _ in range(steps if cold else 1)]
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        if not cold:
            starts[0].record()
        for i in range(steps):
            if flush is not None:
                flush.fill_(float(i))
                starts[i].record()
            self.step(evs[i])
        torch.cuda.synchronize()
        wall = (time.perf_counter() - t0) * 1e3 / steps
        per = []
        for i in range(steps):
            prev = starts[i] if cold else (starts[0] if i == 0 else evs[i - 1][-1])
            row = []
            for e in evs[i]:
                row.append(prev.elapsed_time(e))
                prev = e
            per.append(row)
        return wall, per, preheat


def warm_up(step, warmup: int, warmup_ms: float) -> int:
    """Brings the GPU to its working clock with whole untimed steps for
    warmup_ms of wall time (at least 10 steps; none with warmup_ms 0), then
    runs the warmup untimed steps; returns the pre-heat step count."""
    import torch
    n = 0
    t0 = time.perf_counter()
    while warmup_ms > 0 and (n < 10 or (time.perf_counter() - t0) * 1e3 < warmup_ms):
        for _ in range(10):
            step()
        n += 10
        torch.cuda.synchronize()
    for _ in range(warmup):
        step()
    return n


def _median(v):
    v = sorted(v)
    n = len(v)
    return v[n // 2] if n % 2 else 0.5 * (v[n // 2 - 1] + v[n // 2])


def _slope(xs, ys):
    """Least-squares slope of log y against log x (nan below two points)."""
    if len(xs) < 2:
        return float("nan")
    lx = [math.log(a) for a in xs]
    ly = [math.log(b) for b in ys]
    mx, my = sum(lx) / len(lx), sum(ly) / len(ly)
    num = sum((a - mx) * (b - my) for a, b in zip(lx, ly))
    den = sum((a - mx) ** 2 for a in lx)
    return num / den if den > 0 else float("nan")


def sweep(args):
    import torch
    from paper_2607_12789_amd import inputs
    dev = torch.device("cuda:0")
    rows = []
    for w in inputs.scaling_workloads():
        if args.sweep_only and not any(f == w.name or f == w.name.split("@")[0]
                                       for f in args.sweep_only.split(",")):
            continue
        x = inputs.generate(w)
        r = Runner(w, x, dev)
        wall, per, preheat = r.timed(args.steps, args.warmup, warmup_ms=args.warmup_ms)
        step_ms = _median([sum(p) for p in per])
        k = {name: _median([p[i] for p in per]) for i, name in enumerate(r.stages)}
        qh = w.B * w.H * w.N
        row = {"sweep": w.name, "B": w.B, "H": w.H, "N": w.N, "d": w.d, "M0": w.M0, "Ch": w.Ch,
               "P": w.P, "block_q": w.block_q, "dtype": w.dtype,
               "codes_precompute": w.M0 * (1 + w.Ch), "codes_attention": w.M0 + w.P * w.Ch,
               "ms_median": step_ms, "ms_wall_mean": wall, "qh_per_s": qh / (step_ms * 1e-3),
               "kernels_ms_median": k,
               "steps": args.steps, "warmup": args.warmup,
               "preheat": {"steps": preheat, "ms": args.warmup_ms}}
        rows.append(row)
        print(json.dumps(row), flush=True)
        del r, x
        torch.cuda.empty_cache()
    # slopes against N for each codebook, and against the attention's
    # effective codebook size M0 + P Ch at each N
    by_cb, by_n = {}, {}
    for row in rows:
        by_cb.setdefault(row["sweep"].split("@")[0], []).append(row)
        by_n.setdefault(row["N"], []).append(row)
    summary = {
        "sweep_summary": "log-log slopes of median step time (1 = linear)",
        "slope_vs_N": {cb: round(_slope([r["N"] for r in v], [r["ms_median"] for r in v]), 3)
                       for cb, v in by_cb.items()},
        "slope_vs_N_16k_64k": {
            cb: round(_slope([r["N"] for r in v if r["N"] >= 16384],
                             [r["ms_median"] for r in v if r["N"] >= 16384]), 3)
            for cb, v in by_cb.items()},
        "attention_slope_vs_codes": {
            str(n): round(_slope([r["codes_attention"] for r in v],
                                 [r["kernels_ms_median"]["attention_fwd"] for r in v]), 3)
            for n, v in by_n.items()},
    }
    print(json.dumps(summary), flush=True)


def codebook_bench(args):
    """The codebook step of App. A on the same workload: avq_assign, then
    avq_aggregate on the keys, then avq_codebook_update. One JSON line with
    the per-kernel averages and the update kernel against the HBM peak."""
    import torch
    from paper_2607_12789_amd import avq, inputs
    w = inputs.WORKLOADS[args.workload]
    x = inputs.generate(w)
    dev = torch.device("cuda:0")
    xd = {k: v.to(dev) for k, v in x.items()}
    B, H, N, d, M0, Ch = w.B, w.H, w.N, w.d, w.M0, w.Ch
    Mtot = w.Mtot
    par = torch.empty((B, H, N), dtype=torch.int32, device=dev)
    code = torch.empty_like(par)
    sums = torch.empty((B, H, Mtot, d), dtype=torch.float32, device=dev)
    counts = torch.empty((B, H, Mtot), dtype=torch.int32, device=dev)
    packed = torch.empty((B, H, avq.packed_bytes(w.torch_dtype, M0, Ch, d)), dtype=torch.uint8,
                         device=dev)
    S = torch.zeros((H, Mtot, d), dtype=torch.float32, device=dev)
    Nm = torch.ones((H, Mtot), dtype=torch.float32, device=dev)
    Cp = torch.empty((H, M0, d), dtype=w.torch_dtype, device=dev)
    Cc = torch.empty((H, M0, Ch, d), dtype=w.torch_dtype, device=dev)

    def step(ev=None):
        if ev: ev[0].record()
        avq.assign(xd["K"], xd["Cp"], xd["Cc"], par, code)
        if ev: ev[1].record()
        avq.aggregate(xd["K"], code, M0, Ch, packed, counts, sums)
        if ev: ev[2].record()
        avq.codebook_update(sums, counts, S, Nm, M0, Ch, 0.99, Cp, Cc)
        if ev: ev[3].record()

    preheat = warm_up(step, args.warmup, args.warmup_ms)
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for ev in evs:
        step(ev)
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3 / args.steps
    t = [sum(ev[k].elapsed_time(ev[k + 1]) for ev in evs) / len(evs) for k in range(3)]
    esz = 2 if w.dtype == "bf16" else 4
    # sums and counts read once, S and N read and written, codewords written
    bytes_update = (B * H * Mtot * (d + 1) * 4 + 2 * H * Mtot * (d + 1) * 4
                    + H * Mtot * d * esz)
    achieved = bytes_update / (t[2] * 1e-3) / 1e9
    print(json.dumps({
        "metric": "codebook EMA update step (App. A): assign + key aggregates + update",
        "value": B * H * N / (ms * 1e-3), "unit": "keys*heads/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup,
        "preheat": {"steps": preheat, "ms": args.warmup_ms}, "ms_per_step": ms,
        "higher_is_better": True, "dtype": w.dtype, "data": "synthetic",
        "config": {"workload": f"{w.name}: {w.describe()}", "lambda": 0.99},
        "kernels_ms": {"assign": t[0], "aggregate_keys": t[1], "codebook_update": t[2]},
        "roofline": {"kernel": "avq_codebook_update", "bound": "hbm", "achieved": achieved,
                     "peak": 8000.0, "unit": "GB/s", "frac": achieved / 8000.0, "traffic": None,
                     "bytes_per_launch": bytes_update},
    }), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=10,
                    help="untimed warm-up steps, after the pre-heat")
    ap.add_argument("--warmup-ms", type=float, default=200.0,
                    help="wall time of the pre-heat: untimed steps before the warm-up steps "
                         "that bring the GPU clock up (0: none)")
    ap.add_argument("--workload", default="c4")
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="least wall time the oracle baseline runs for")
    ap.add_argument("--cpu-max-passes", type=int, default=8)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-threads", type=int, default=0,
                    help="threads of the oracle baseline (0: all host cores)")
    ap.add_argument("--cold", action="store_true",
                    help="before every step, overwrite a 1 GiB buffer (four times the "
                         "256 MB last-level cache) outside the timed events, so that each "
                         "step starts with inputs in HBM only; the step time is then the "
                         "sum of the event-timed entry points")
    ap.add_argument("--calib-copy-mib", type=int, default=0,
                    help="also launch one plain device copy of this many MiB (counter calibration)")
    ap.add_argument("--unfused-precompute", action="store_true",
                    help="run the precompute as avq_assign then avq_aggregate instead of the "
                         "one-pass avq_assign_aggregate")
    ap.add_argument("--tiled-importance", action="store_true",
                    help="use the App. B importance (one parent sweep) instead of the exact one")
    ap.add_argument("--query-order", choices=["token", "gilbert", "random"], default="token",
                    help="order of the queries: token order, or the tokens as a square grid "
                         "along a Gilbert curve, or a random permutation")
    ap.add_argument("--top-p", type=int, default=None,
                    help="run the workload with this P instead of its own (a diagnostic of the "
                         "attention's phases: 0 leaves the parent sweep and the output alone); "
                         "the line then names the override and carries no traffic figure")
    ap.add_argument("--codebook-update", action="store_true",
                    help="time the codebook EMA step (App. A) instead")
    ap.add_argument("--sweep", action="store_true",
                    help="run the sequence-length scaling sweep instead")
    ap.add_argument("--sweep-only", default="",
                    help="comma-separated sweep workloads (e.g. vq256@N=65536) or codebooks "
                         "(e.g. avq64/8/8) to run")
    args = ap.parse_args()

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU only: this build has no multi-GPU path "
              f"(asked for --gpus {args.gpus}, WORLD_SIZE={world}).", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2607_12789_amd import avq, inputs

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    if args.sweep:
        sweep(args)
        return
    if args.codebook_update:
        codebook_bench(args)
        return
    w = inputs.WORKLOADS[args.workload]
    x = inputs.generate(w)
    name = w.name
    if args.top_p is not None:  # the same inputs, another number of selected parents
        if not 0 <= args.top_p <= w.M0:
            print(f"--top-p must lie in [0, M0 = {w.M0}]", file=sys.stderr)
            sys.exit(2)
        w = dataclasses.replace(w, P=args.top_p)
        name = f"{w.name} with P overridden to {w.P}"
    dev = torch.device("cuda:0")
    B, H, N, d, M0, Ch, P = w.B, w.H, w.N, w.d, w.M0, w.Ch, w.P
    order = None
    if args.query_order == "gilbert":
        side = int(round(math.sqrt(w.N)))
        if side * side != w.N:
            print(f"--query-order gilbert needs a square number of tokens (N={w.N})",
                  file=sys.stderr)
            sys.exit(2)
        order = avq.gilbert_order(side, side)[0]
    elif args.query_order == "random":
        order = torch.randperm(w.N, generator=torch.Generator().manual_seed(0)).to(torch.int32)
    runner = Runner(w, x, dev, args.tiled_importance, order, not args.unfused_precompute)
    ms_per_step, per, preheat = runner.timed(args.steps, args.warmup, args.cold, args.warmup_ms)
    if args.cold:  # the wall clock includes the fills: the steps are the events
        ms_per_step = sum(sum(p) for p in per) / max(len(per), 1)
    # per-entry-point average duration over the timed steps
    stage_ms = {name: sum(p[i] for p in per) / max(len(per), 1)
                for i, name in enumerate(runner.stages)}
    t_attn = stage_ms["attention_fwd"]
    if args.calib_copy_mib > 0:
        n = args.calib_copy_mib * (1 << 20) // 4
        src = torch.ones(n, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()

    qh = B * H * N
    flops_attn = 4.0 * d * (M0 + P * Ch) * qh
    achieved = flops_attn / (t_attn * 1e-3) / 1e12
    # the MFMA peak of the kernel's own type: bf16 2.5 PFLOP/s, fp32 157.3 TFLOP/s
    peak = PEAK_BF16_TFLOPS if w.dtype == "bf16" else PEAK_F32_TFLOPS
    traffic = (None if (args.tiled_importance or order is not None or args.top_p is not None)
               else read_traffic())
    # the precompute against HBM: K and V read once, the codebooks read once per
    # head, parent indices, codes, counts and packed aggregates written once
    esz = 2 if w.dtype == "bf16" else 4
    Mtot = M0 * (1 + Ch)
    bytes_pre = (2 * qh * d * esz + H * M0 * (1 + Ch) * d * esz
                 + B * H * (2 * N * 4 + Mtot * 4 + avq.packed_bytes(x["K"].dtype, M0, Ch, d)))
    t_pre = sum(v for k, v in stage_ms.items() if k != "attention_fwd")
    pre_gbs = bytes_pre / (t_pre * 1e-3) / 1e9
    line = {
        "metric": METRIC,
        "value": qh / (ms_per_step * 1e-3),
        "unit": UNIT,
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "preheat": {"steps": preheat, "ms": args.warmup_ms},
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if w.dtype == "bf16" else "f32",
        "data": "synthetic",
        "config": {"workload": f"{name}: {w.describe()}", "B": B, "H": H, "N": N, "d": d,
                   "M0": M0, "Ch": Ch, "P": P, "block_q": w.block_q,
                   "importance": "tiled (App. B, 64-parent tiles)" if args.tiled_importance
                   else "exact", "query_order": args.query_order,
                   "precompute": "avq_assign + avq_aggregate" if args.unfused_precompute
                   else "avq_assign_aggregate (Alg. 1, one pass)",
                   "caches": "cold (1 GiB fill before each step)" if args.cold else "warm"},
        "kernels_ms": stage_ms,
        "ms_per_step_median": _median([sum(p) for p in per]),
        "roofline": {"kernel": ("avq_attention_fwd_ordered" if order is not None else
                                "avq_attention_fwd_tiled" if args.tiled_importance
                                else "avq_attention_fwd"), "bound": "mfma", "achieved": achieved,
                     "peak": peak, "unit": "TFLOP/s",
                     "frac": achieved / peak, "traffic": traffic,
                     "flops_per_launch": flops_attn},
        "precompute_roofline": {"kernels": [k for k in stage_ms if k != "attention_fwd"],
                                "bound": "hbm", "achieved": pre_gbs, "peak": 8000.0,
                                "unit": "GB/s", "frac": pre_gbs / 8000.0,
                                "bytes_per_step": bytes_pre},
    }
    if not args.no_cpu_baseline:
        if args.cpu_threads > 0:
            import oracle
            oracle.set_num_threads(args.cpu_threads)
        line["cpu_baseline"] = cpu_baseline(x, w, args.cpu_seconds, args.cpu_max_passes)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
