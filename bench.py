"""Throughput of the AVQ-Attention forward pass on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W]

One step is the whole forward pass over one batch of synthetic inputs
already resident in HBM: avq_assign -> avq_aggregate -> avq_attention_fwd.
The workload is the N = 16384 one (B=2, H=16, d=128, M0=256 parents with 8
children each, P=32, query block 128, bf16). Prints one JSON line:

* value: query-token*heads per second of the whole step, B*H*N / t_step;
* roofline: the fused attention kernel (the dominant one) against the bf16
  MFMA peak, its algorithmic flops 4 d (M0 + P Ch) per query-head divided by
  its average launch duration over the timed steps (HIP events bracketing
  each launch, on the launch stream); traffic is the
  HBM bytes per launch from the committed rocprofv3 counter summary, or null
  if the kernel source changed since those counters were taken;
* cpu_baseline: the fp64 oracle timed on the host cores, whole passes over
  the same workload repeated for at least --cpu-seconds.
"""
from __future__ import annotations

import argparse
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
KERNEL_SRC = ROOT / "paper_2607_12789_amd" / "csrc" / "avq_attention.hip"
TRAFFIC_SUMMARY = ROOT / "profiles" / "attention_fwd_c4_traffic.md"


def kernel_hash() -> str:
    h = hashlib.sha256()
    for name in ("avq_attention.hip", "avq_common.hpp", "avq_packed.hpp"):
        h.update((KERNEL_SRC.parent / name).read_bytes())
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


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="c4")
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="least wall time the oracle baseline runs for")
    ap.add_argument("--cpu-max-passes", type=int, default=8)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--calib-copy-mib", type=int, default=0,
                    help="also launch one plain device copy of this many MiB (counter calibration)")
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
    w = inputs.WORKLOADS[args.workload]
    x = inputs.generate(w)
    dev = torch.device("cuda:0")
    xd = {k: v.to(dev) for k, v in x.items()}
    B, H, N, d, M0, Ch, P = w.B, w.H, w.N, w.d, w.M0, w.Ch, w.P
    par = torch.empty((B, H, N), dtype=torch.int32, device=dev)
    code = torch.empty_like(par)
    packed = torch.empty((B, H, avq.packed_bytes(w.torch_dtype, M0, Ch, d)), dtype=torch.uint8,
                         device=dev)
    counts = torch.empty((B, H, w.Mtot), dtype=torch.int32, device=dev)
    Y = torch.empty_like(xd["Q"])

    def step(ev=None):
        # ev: four events bracketing the three launches (HIP events on the
        # stream the kernels are launched on, which is torch's current one)
        if ev: ev[0].record()
        avq.assign(xd["K"], xd["Cp"], xd["Cc"], par, code)
        if ev: ev[1].record()
        avq.aggregate(xd["V"], code, M0, Ch, packed, counts)
        if ev: ev[2].record()
        avq.attention_fwd(xd["Q"], xd["Cp"], xd["Cc"], packed, P, w.block_q, Y=Y)
        if ev: ev[3].record()

    for _ in range(args.warmup):
        step()
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        step(evs[i])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_per_step = wall * 1e3 / args.steps

    # per-kernel average launch duration over the timed steps
    def avg_ms(a, b):
        return sum(ev[a].elapsed_time(ev[b]) for ev in evs) / max(len(evs), 1)

    t_assign, t_agg, t_attn = avg_ms(0, 1), avg_ms(1, 2), avg_ms(2, 3)
    if args.calib_copy_mib > 0:
        n = args.calib_copy_mib * (1 << 20) // 4
        src = torch.ones(n, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()

    qh = B * H * N
    flops_attn = 4.0 * d * (M0 + P * Ch) * qh
    achieved = flops_attn / (t_attn * 1e-3) / 1e12
    traffic = read_traffic()
    line = {
        "metric": METRIC,
        "value": qh / (ms_per_step * 1e-3),
        "unit": UNIT,
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if w.dtype == "bf16" else "f32",
        "data": "synthetic",
        "config": {"workload": f"{w.name}: {w.describe()}", "B": B, "H": H, "N": N, "d": d,
                   "M0": M0, "Ch": Ch, "P": P, "block_q": w.block_q},
        "kernels_ms": {"assign": t_assign, "aggregate": t_agg, "attention_fwd": t_attn},
        "roofline": {"kernel": "avq_attention_fwd", "bound": "mfma", "achieved": achieved,
                     "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                     "frac": achieved / PEAK_BF16_TFLOPS, "traffic": traffic,
                     "flops_per_launch": flops_attn},
    }
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(x, w, args.cpu_seconds, args.cpu_max_passes)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
