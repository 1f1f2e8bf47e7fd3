"""Benchmark: WaveRNN sampling throughput on one MI355X.

One bench step = one ``wavernn_sample`` call that generates a whole synthetic
utterance (Dense WaveRNN-896, batch 1, 24,000 samples = 1 s of 24 kHz audio):
the full per-sample hot path (GRU of Eq. 2, coarse head, coarse draw, fine
half, fine head, fine draw) 24,000 times inside one persistent kernel.
Prints one JSON line.  ``value`` is audio samples per second with inputs
resident in HBM; ``us_per_sample`` is the mean time of one sampling step.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "audio samples/sec (xreal-time @24kHz) and us/step, WaveRNN-896 batch 1"
PAPER_SAMPLES_PER_S = 96000.0   # WaveRNN-896 batch 1 on a P100 (Sec. 2.1); context, other hardware
HBM_PEAK_GBS = 8000.0
LDS_BYTES_PER_CLK_CU = 128
CLOCK_GHZ = 2.4


def weight_bytes_per_step(w: dict) -> int:
    """Algorithmic bytes one sampling step must read: every weight once (bf16)."""
    H = w["H"]
    Hh = H // 2
    nR = int((w["R"] != 0).sum()) if w.get("mask") is not None else 3 * H * H
    n = nR + 2 * (Hh * Hh + 256 * Hh)
    if w.get("Wx") is not None:          # subscale context projection
        n += int(w["Wx"].size)
    bytes_per = 2 if w.get("bf16", True) else 4
    return n * bytes_per


# kernel that serves each path of wavernn_model_path
KERNEL_OF = {"persistent": "wr_persist_kernel", "block-sparse": "wr_sparse_kernel", "batched": "wr_batch_kernel",
             "single-workgroup": "wr_small_kernel"}


def kernel_source_digest() -> str:
    """Digest of every kernel and host source of the library (any change voids old counters)."""
    import hashlib
    h = hashlib.sha256()
    d = os.path.join(ROOT, "paper_1802_08435_amd", "csrc")
    for f in sorted(os.listdir(d)):
        if f.endswith((".hip", ".h")):
            with open(os.path.join(d, f), "rb") as fh:
                h.update(f.encode() + fh.read())
    return h.hexdigest()[:16]


def measured_traffic(kernel: str, workload: str):
    """HBM bytes per launch from the committed rocprofv3 --pmc summary of this kernel and workload,
    or None when the library sources changed since the counters were taken."""
    path = os.path.join(ROOT, "profiles", f"{kernel}_{workload}.md")
    if not os.path.exists(path):
        return None
    text = open(path).read()
    i = text.find("```json")
    if i < 0:
        return None
    d = json.loads(text[i + 7:text.index("```", i + 7)])
    if d.get("kernel_source_sha256_16") != kernel_source_digest():
        return None
    return d["fetch_bytes_per_launch"] + d["write_bytes_per_launch"]


def cpu_baseline(w: dict, T: int, feat, budget_s: float = 12.0) -> dict:
    """The oracle as it stands, single-threaded on the host, on a bounded prefix."""
    import numpy as np
    from oracle import oracle
    W = oracle.Weights.from_dict(w, bf16=w.get("bf16", False))
    t = time.perf_counter()
    oracle.run(W, 1, 50, feat=feat[:1], seed=1)
    per = (time.perf_counter() - t) / 50
    n = int(max(50, min(T, budget_s / max(per, 1e-9))))
    t = time.perf_counter()
    oracle.run(W, 1, n, feat=feat[:1], seed=1)
    dt = time.perf_counter() - t
    return {"value": round(n / dt, 2), "unit": "samples/s", "cores": 1, "kind": "oracle",
            "sample": f"first {n} of the {T} samples of one utterance, single-threaded C oracle (gcc -O2)"}


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--config", default="dense896")
    ap.add_argument("--samples", type=int, default=0, help="override samples per utterance")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="MIB",
                    help="only run a plain device-to-device copy of MIB MiB (HBM counter calibration) and exit")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py: this build runs on one GPU; --gpus {args.gpus} is not supported "
              "(utterances are independent: more GPUs would each run their own).", file=sys.stderr)
        return 2

    import numpy as np
    import torch
    from paper_1802_08435_amd import synth, wavernn

    torch.cuda.set_device(0)
    if args.calibrate_copy:
        n = args.calibrate_copy << 20
        src = torch.ones(n // 4, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes_read": n, "copy_bytes_written": n, "launches": 3}), flush=True)
        return 0
    w = synth.preset(args.config)
    S, T = w["streams"], args.samples or w["samples"]
    r_format = {None: "dense", (4, 4): "bsr4x4", (16, 1): "bsr16x1"}[w["block"]]
    m = wavernn.Model(w, dtype="bf16" if w["bf16"] else "f32", r_format=r_format, max_streams=S)
    path, grid, block = m.path(S)
    feat_np = synth.features(S, T, per_stream_seed=S > 1)
    feat = torch.from_numpy(feat_np).cuda()
    out = torch.empty(S, T, dtype=torch.uint16, device="cuda")
    stream = torch.cuda.current_stream()
    for i in range(args.warmup):
        m.sample(T, cond=feat, seed=1 + i, n_streams=S, out=out)
    torch.cuda.synchronize()
    m.device_status()
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        evs[i][0].record(stream)
        m.sample(T, cond=feat, seed=100 + i, n_streams=S, out=out)
        evs[i][1].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    m.device_status()
    call_ms = [a.elapsed_time(b) for a, b in evs]
    # synchronization floor: the same grid and exchanged words per step, no arithmetic
    floor_us = m.sync_floor(T // w["B"]) if path in ("persistent", "block-sparse") else None
    ms = float(np.mean(call_ms))
    samples = S * T
    value = samples * args.steps / wall
    us_per_sample_step = ms * 1000.0 / (T // w["B"])
    wb = weight_bytes_per_step(w)
    steps_per_launch = T // w["B"]
    achieved = wb * steps_per_launch / (ms / 1000.0) / 1e9
    ncu = grid
    lds_peak = ncu * LDS_BYTES_PER_CLK_CU * CLOCK_GHZ
    kname = KERNEL_OF.get(path, path)
    tb = measured_traffic(kname, args.config) if T == w["samples"] and S == w["streams"] else None
    traffic = None if tb is None else round(tb / (ms / 1000.0) / 1e9, 2)
    line = {
        "metric": METRIC,
        "value": round(value, 1),
        "unit": "samples/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": round(value / PAPER_SAMPLES_PER_S, 3) if args.config == "dense896" else None,
        "dtype": "bf16" if w["bf16"] else "f32",
        "data": "synthetic (seeded N(0,1/fan_in) weights, N(0,1) conditioning frames)",
        "config": {"workload": f"{args.config}: H={w['H']}, B={w['B']}, {S} utterance(s) x {T} samples",
                   "weights": "bf16" if w["bf16"] else "f32", "kernel": path, "grid": grid, "block": block},
        "us_per_sample": round(us_per_sample_step, 4),
        "x_realtime": round(value / 24000.0, 3),
        "call_ms_min": round(min(call_ms), 4),
        "sync_floor": None if floor_us is None else {
            "us_per_step": round(floor_us, 4), "frac_of_step": round(floor_us / us_per_sample_step, 4)},
        "roofline": {"bound": "hbm", "achieved": round(achieved, 2), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(achieved / HBM_PEAK_GBS, 5), "traffic": traffic,
                     "kernel": kname, "bytes_per_step": wb, "steps_per_launch": steps_per_launch,
                     "lds_frac": round(achieved / lds_peak, 5)},
    }
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(w, T, feat_np)
    print(json.dumps(line), flush=True)
    m.close()
    torch.cuda.synchronize()
    return 0


if __name__ == "__main__":
    sys.exit(main())
