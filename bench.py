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


def weight_bytes_per_step(w: dict) -> int:
    """Algorithmic bytes one sampling step must read: every weight once (bf16)."""
    H = w["H"]
    Hh = H // 2
    if w.get("fused"):                   # R, four Q x Q first layers, four 32 x Q nibble layers
        Q = H // 4
        return 2 * (3 * H * H + 4 * Q * Q + 4 * 32 * Q)
    nR = int((w["R"] != 0).sum()) if w.get("mask") is not None else 3 * H * H
    n = nR + 2 * (Hh * Hh + 256 * Hh)
    if w.get("Wx") is not None:          # subscale context projection
        n += int(w["Wx"].size)
    bytes_per = 2 if w.get("bf16", True) else 4
    return n * bytes_per


# kernel that serves each path of wavernn_model_path
KERNEL_OF = {"persistent": "wr_persist_kernel", "block-sparse": "wr_sparse_kernel", "batched": "wr_batch_kernel",
             "single-workgroup": "wr_small_kernel", "concurrent": "wr_persist_kernel", "fused": "wr_fused_kernel"}


# source file of each kernel (the digest covers it and the headers it includes)
KERNEL_SOURCE = {"wr_persist_kernel": "wr_persist.hip", "wr_sparse_kernel": "wr_persist.hip",
                 "wr_fused_kernel": "wr_fused.hip", "wr_batch_kernel": "wr_batch.hip", "wr_small_kernel": "wr_small.hip"}


def kernel_source_digest(kernel: str) -> str:
    """Digest of the device sources a kernel is compiled from: its .hip file and every header it
    includes, directly or not (any change voids the counters taken on it)."""
    import hashlib
    import re
    d = os.path.join(ROOT, "paper_1802_08435_amd", "csrc")
    todo, seen = [KERNEL_SOURCE[kernel]], set()
    while todo:
        f = todo.pop()
        if f in seen or not os.path.exists(os.path.join(d, f)):
            continue
        seen.add(f)
        todo += re.findall(r'#include "([^"]+)"', open(os.path.join(d, f)).read())
    h = hashlib.sha256()
    for f in sorted(seen):
        with open(os.path.join(d, f), "rb") as fh:
            h.update(f.encode() + fh.read())
    return h.hexdigest()[:16]


def measured_traffic(kernel: str, workload: str):
    """HBM bytes per call (its launches of the kernel) from the committed rocprofv3 --pmc summary of
    this kernel and workload, or None when the kernel's sources changed since the counters were taken."""
    path = os.path.join(ROOT, "profiles", f"{kernel}_{workload}.md")
    if not os.path.exists(path):
        return None
    text = open(path).read()
    i = text.find("```json")
    if i < 0:
        return None
    d = json.loads(text[i + 7:text.index("```", i + 7)])
    if d.get("kernel_source_sha256_16") != kernel_source_digest(kernel):
        return None
    return (d["fetch_bytes_per_launch"] + d["write_bytes_per_launch"]) * d.get("launches_per_call", 1)


def cpu_baseline(w: dict, T: int, feat, budget_s: float = 12.0) -> dict:
    """The oracle as it stands, single-threaded on the host, on a bounded prefix."""
    import numpy as np
    from oracle import oracle
    if w.get("fused"):
        keys = ("R", "I", "b", "O1", "b1", "O2", "b2", "Wc")
        d = {k: (None if w.get(k) is None else oracle.bf16_round(w[k])) for k in keys}
        d.update(H=w["H"], F=w["F"])
        run = lambda n: oracle.fused_run(d, 1, n, feat=feat[:1], seed=1, frame_len=w["frame_len"])
        t = time.perf_counter()
        run(48)
        per = (time.perf_counter() - t) / 48
        n = int(max(48, min(T, budget_s / max(per, 1e-9)))) // 2 * 2
        t = time.perf_counter()
        run(n)
        dt = time.perf_counter() - t
        return {"value": round(n / dt, 2), "unit": "samples/s", "cores": 1, "host_cores": os.cpu_count(),
                "kind": "oracle",
                "sample": f"first {n} of the {T} samples of one utterance, single-threaded C oracle (gcc -O2)"}
    W = oracle.Weights.from_dict(w, bf16=w.get("bf16", False))
    B = w.get("B", 1)                                    # subscale: whole rows of B samples
    n0 = 48 // B * B or B
    t = time.perf_counter()
    oracle.run(W, 1, n0, feat=feat[:1], seed=1)
    per = (time.perf_counter() - t) / n0
    n = int(max(n0, min(T, budget_s / max(per, 1e-9)))) // B * B
    t = time.perf_counter()
    oracle.run(W, 1, n, feat=feat[:1], seed=1)
    dt = time.perf_counter() - t
    return {"value": round(n / dt, 2), "unit": "samples/s", "cores": 1, "host_cores": os.cpu_count(),
            "kind": "oracle",
            "sample": f"first {n} of the {T} samples of one utterance, single-threaded C oracle (gcc -O2)"}


BF16_MFMA_PEAK_TFLOPS = 2500.0   # dense bf16 matrix-core peak of the MI355X


def cnn_flops_per_row(w: dict) -> int:
    """Algorithmic FLOPs of the conditioning CNN per row of one sub-tensor (2 per multiply-add)."""
    c = w["cnn"]
    Rc, B, Dx = c["Win"].shape[0], w["B"], c["Wp"].shape[0]
    L = int(c["layers"])
    Cc = c["bc"].shape[1] if L else 0
    return 2 * (2 * B * Rc + L * (3 * Rc * Cc + Cc * Rc) + Rc * Dx)


def cnn_table(m, w: dict, seq, reps: int = 5) -> dict:
    """The conditioning CNN over the whole generated utterance(s), timed with
    HIP events on the launch stream: its matrix-core roofline (bf16 dense peak)."""
    import numpy as np
    import torch
    st = torch.cuda.current_stream()
    m.ctx_cnn(seq)
    torch.cuda.synchronize()
    ms = []
    for _ in range(reps):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(st)
        m.ctx_cnn(seq)
        b.record(st)
        torch.cuda.synchronize()
        ms.append(a.elapsed_time(b))
    m.device_status()
    rows = seq.shape[0] * seq.shape[1]                   # every row of every sub-tensor: S x B x N / B
    flops = cnn_flops_per_row(w) * rows
    t = float(np.median(ms)) / 1000.0
    return {"rows": rows, "ms_median": round(float(np.median(ms)), 4), "gflop": round(flops / 1e9, 2),
            "bound": "mfma", "achieved": round(flops / t / 1e12, 2), "peak": BF16_MFMA_PEAK_TFLOPS,
            "unit": "TFLOP/s", "frac": round(flops / t / 1e12 / BF16_MFMA_PEAK_TFLOPS, 4),
            "kernel": "wr_cnn_gemm (all 22 GEMMs of a table, plus wr_cnn_input)"}


# In-kernel timestamps (trace slot -> phase end) of the step loop of head 0
# (group 0 for the batched kernel), recorded by wavernn_set_trace.
PHASES = {
    "persistent": [(1, "coarse gates (Eq. 2, with f_{t-1}) done, own y_c slice published"),
                   (2, "O1 rows + relu"), (3, "O2 columns: partial coarse logits published"),
                   (15, "coarse partials of all heads received (draw wave)"),
                   (16, "c_t drawn (draw wave)"), (5, "barrier: c_t known to all waves"),
                   (6, "fine gates (with c_t) done, own y_f slice published"), (7, "O3 rows + relu"),
                   (8, "O4 columns: partial fine logits published"),
                   (17, "fine partials of all heads received (draw wave)"), (18, "f_t drawn (draw wave)"),
                   (10, "next step's coarse gate words received (end of step)")],
    "batched": [(11, "coarse gate words received"), (1, "coarse gates done, y_c of the group exchanged"),
                (3, "O1/O2: partial coarse logits published"), (4, "owned vectors' coarse partials summed"),
                (5, "c_t drawn"), (12, "fine gate words (groups of 2 and 4: read with the coarse ones) and classes received"),
                (6, "fine gates done, y_f of the group exchanged"), (8, "O3/O4: partial fine logits published"),
                (9, "owned vectors' fine partials summed"), (10, "f_t drawn (end of step)")],
}
PHASES["block-sparse"] = [(1, "coarse gates (Eq. 2, with f_{t-1}) done, own y_c slice published"),
                          (2, "O1 rows + relu"), (3, "O2 columns: partial coarse logits published"),
                          (15, "coarse partials of all heads received"), (4, "barrier"),
                          (16, "c_t drawn (draw wave)"), (5, "barrier: c_t known to all waves"),
                          (6, "fine gates (with c_t) done, own y_f slice published"), (7, "O3 rows + relu"),
                          (8, "O4 columns: partial fine logits published"),
                          (17, "fine partials of all heads received"), (9, "barrier"), (18, "f_t drawn (draw wave)"),
                          (10, "next step's coarse gate words received (end of step)")]
PHASES["fused"] = [(1, "coarse gates (last f of both sub-tensors) done, own y_c slice published"),
                   (3, "coarse MLPs: 64 partial nibble logits published"),
                   (16, "partials of all heads summed, 4 coarse nibbles drawn (draw wave)"),
                   (5, "barrier: coarse bytes known to all waves"),
                   (6, "fine gates (own coarse byte) done, own y_f slice published"),
                   (8, "fine MLPs: partial nibble logits published"),
                   (18, "4 fine nibbles drawn (draw wave)"), (10, "next step's coarse gate words received (end of step)")]


# Stamps of other workgroups of the same step (µs from head 0's step start),
# reported beside the chain above.
SIDE = {"persistent": [(23, "mirror 0: its coarse rows' products with y_f published"),
                       (11, "unit 0: y_f in, fine rows' products started"),
                       (12, "unit 0: fine rows' words of the next step published")]}
SIDE["fused"] = SIDE["persistent"]


def phases(m, w, path: str, S: int, feat, n_steps: int) -> dict:
    """Median per-phase timestamps of one traced launch of n_steps steps (the
    first and last eighth left out)."""
    import numpy as np
    import torch
    B = w["B"]
    T = n_steps * B
    skip = n_steps // 8
    buf = torch.zeros(n_steps, 32, dtype=torch.int64, device="cuda")
    m.set_trace(buf)
    m.sample(T, cond=feat, seed=5, n_streams=S)
    torch.cuda.synchronize()
    m.set_trace(None)
    m.device_status()
    tr = buf.cpu().numpy()[skip:n_steps - skip].astype(np.int64)
    step_ns = np.diff(tr[:, 0]) * 10.0                    # 100 MHz clock
    rel = (tr - tr[:, [0]]) * 10.0
    out, prev = [], 0.0
    for slot, name in PHASES[path]:
        if (tr[:, slot] == 0).any():
            continue
        t = float(np.median(rel[:, slot]))
        out.append({"slot": slot, "phase": name, "end_ns": round(t), "took_ns": round(t - prev)})
        prev = t
    side = []
    for slot, name in SIDE.get(path, []):
        if (tr[:, slot] == 0).any():
            continue
        # unit stamps 11 and 12 are recorded under the step they serve (t + 1)
        col = rel[1:, slot] + (tr[1:, 0] - tr[:-1, 0]) * 10.0 if slot in (11, 12) else rel[:, slot]
        side.append({"slot": slot, "event": name, "at_ns": round(float(np.median(col)))})
    return {"phases": out, "side": side, "step_ns_median": round(float(np.median(step_ns))),
            "step_ns_p10": round(float(np.percentile(step_ns, 10))),
            "step_ns_p90": round(float(np.percentile(step_ns, 90))), "traced_steps": int(len(step_ns))}


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
    ap.add_argument("--placement", type=int, default=None, metavar="K",
                    help="fix the batch-1 launches' placement to candidate K (wavernn_tune's numbering) instead "
                         "of tuning it (-1: the default placement)")
    ap.add_argument("--phases", action="store_true",
                    help="only time the phases of one traced launch (in-kernel timestamps) and print them")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py: the benchmark runs on one GPU; --gpus {args.gpus} is not supported "
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
    r_format = {None: "dense", (4, 4): "bsr4x4", (16, 1): "bsr16x1"}[w.get("block")]
    m = wavernn.Model(w, dtype="bf16" if w["bf16"] else "f32", r_format=r_format, max_streams=S)
    path, grid, block = m.path(S)
    placement = None
    if path in ("persistent", "block-sparse", "fused"):   # batch-1 launches: pick the XCDs of heads and units
        if args.placement is None:
            tu = m.tune(n_steps=2048, rounds=2)
            k, us = tu["chosen"], tu["us_per_step"]
            placement = {"candidate": k, "tuned": True, "tune_us_per_step": round(us[k], 4),
                         "default_us_per_step": round(us[0], 4), "candidates_timed": sum(1 for x in us if x > 0)}
        else:
            m.set_placement(args.placement)
            k = max(args.placement, 0)
            placement = {"candidate": k, "tuned": False}
        placement.update(heads_xcd=k // 8, units_xcd="all" if k % 8 == k // 8 else k % 8)
        path, grid, block = m.path(S)
    feat_np = synth.features(S, T, per_stream_seed=S > 1)
    feat = torch.from_numpy(feat_np).cuda()
    out = torch.empty(S, T, dtype=torch.uint16, device="cuda")
    stream = torch.cuda.current_stream()
    if args.phases:
        if path not in PHASES or w.get("cnn") is not None:   # no phase stamps / tracing switched off
            why = ("tracing is switched off for CNN-conditioned calls" if w.get("cnn") is not None
                   else "this kernel has no phase stamps")
            print(json.dumps({"workload": args.config, "kernel": KERNEL_OF.get(path, path), "phases": None,
                              "why": why}), flush=True)
            m.close()
            return 0
        m.sample(T, cond=feat, seed=1, n_streams=S, out=out)
        ph = phases(m, w, path, S, feat, min(T // w["B"], 4000))
        print(json.dumps({"workload": args.config, "kernel": KERNEL_OF.get(path, path), **ph}), flush=True)
        m.close()
        return 0
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
    # (the floor kernel gathers the fused heads' 64 nibble partials with every thread; it is not a lower
    # bound for the fused kernel's one-wave gather, so fused models report none)
    floor_us = (m.sync_floor(T // w["B"]) if path in ("persistent", "block-sparse", "batched", "concurrent")
                and w.get("cnn") is None else None)
    # teacher-forced scoring of the last sampled utterance (logits of both heads and the NLL)
    score = None
    if w["B"] == 1 and path in ("persistent", "concurrent", "batched"):   # dense models: the recurrence kernels
        m.score(out, cond=feat)
        torch.cuda.synchronize()
        sm = []
        for _ in range(3):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(stream)
            m.score(out, cond=feat)
            b.record(stream)
            torch.cuda.synchronize()
            sm.append(a.elapsed_time(b))
        m.device_status()
        smed = float(np.median(sm))
        score = {"call_ms_median": round(smed, 4), "samples_per_s": round(S * T / (smed / 1000.0), 1),
                 "utterances": S, "us_per_step": round(smed * 1000.0 / T, 4),
                 "kernels": ("wr_score_kernel (one grid per utterance)" if S <= 4 else
                             "wr_score_multi (8 utterances per grid, 4 grids side by side)") +
                            " + wr_cnn_gemm (output layers over all steps) + wr_score_nll"}
    ms = float(np.mean(call_ms))
    samples = S * T
    value = samples * args.steps / wall
    F, A = w.get("F", -1), w.get("A", 0)               # subscale horizon and lead: (B - 1)(F + 1 + A) more steps
    steps_per_launch = T // w["B"] + ((w["B"] - 1) * (F + 1 + A) if F >= 0 else 0)   # fused 2x: T / 2 + F + 1
    us_per_sample_step = ms * 1000.0 / steps_per_launch
    wb = weight_bytes_per_step(w)
    achieved = wb * steps_per_launch / (ms / 1000.0) / 1e9
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
        "call_ms_median": round(float(np.median(call_ms)), 4),
        "placement": placement,
        "teacher_forced_score": score,
        "sync_floor": None if floor_us is None else {
            "us_per_step": round(floor_us, 4), "frac_of_step": round(floor_us / us_per_sample_step, 4)},
        "limiter": ("cross-CU exchange latency: the weights stay in VGPRs and LDS, so the HBM roofline below is "
                    "the weights' algorithmic bytes per step; the synchronization floor of the same launch "
                    f"(its exchanges and waits, no arithmetic) takes {floor_us / us_per_sample_step:.0%} of the step")
                   if floor_us is not None else None,
        "roofline": {"bound": "hbm", "achieved": round(achieved, 2), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(achieved / HBM_PEAK_GBS, 5), "traffic": traffic,
                     "kernel": kname, "bytes_per_step": wb, "steps_per_launch": steps_per_launch},
    }
    if w.get("cnn") is not None:
        line["cnn_table"] = cnn_table(m, w, out)
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(w, T, feat_np)
    print(json.dumps(line), flush=True)
    m.close()
    torch.cuda.synchronize()
    return 0


if __name__ == "__main__":
    sys.exit(main())
