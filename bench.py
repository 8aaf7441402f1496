"""Benchmark of the GoCkpt hot path on one MI355X.

    python bench.py [--steps 8] [--warmup 8] [--workload llama13b_k32] [--tfb-ms auto] [--shard I/P]

A step is one training step with a save window open: the forward/backward
stand-in (a kernel holding the device for T_fb, its backward part shortened
by the gradient generation's measured time), the gradient generation
(writes the 16-bit gradient buffer, standing in for the backward's output),
then ``gockpt_step``: prepass, finalize (skip decision, loss scaler, step
scalars), fused AdamW update + pack of the step's part and of the gradients
of the parts already sent, and the D2H copies of that pack queued on the copy stream,
where they overlap the next step.  All inputs are resident in HBM before the
timed region.  Windows of K steps follow each other; the host restore of a
window runs outside the timed region and is reported on its own.  The
default workload is the largest one a single GPU holds (Llama-style 13B,
K = 32).

    python bench.py --summarize-traffic FETCH_CSV WRITE_CSV BENCH_JSON

writes profiles/fused_kernel_<workload>_traffic.{json,md} from two rocprofv3
counter runs of this bench (FETCH_SIZE, WRITE_SIZE) and the JSON line one of
them printed.

One JSON line on stdout:
  value            fused step+pack HBM GB/s: algorithmic bytes of the prepass
                   (2 B/element) and of the update+pack (28 B/element + 12 B
                   per element of the step's part + 2 B per gradient sent)
                   over the device time of those kernels, from HIP events on
                   the compute stream, summed over the timed steps
  d2h_gbs          bytes copied to the host / copy-stream busy time, next to
                   the host-link D2H rate measured in the same run
  stall_ms_per_step  checkpoint stall per window step: compute-stream time of
                   the K window steps and the step after them (no host drain
                   inside) minus the same span of K + 1 plain steps taken
                   just before it, divided by K; median over 3 such pairs
  roofline         the fused update+pack kernel alone against 8 TB/s
  cpu_baseline     the oracle on this host's cores, on a bounded sample
"""
from __future__ import annotations

import argparse
import ctypes
import json
import os
import statistics
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "fused step+pack HBM GB/s (% of peak); D2H GB/s; stall ms/step"
HBM_PEAK_GBS = 8000.0
RECORD_BYTES = 64
RING_PLANS = {"query": 0, "host": 1, "device": 2}


def log(msg: str) -> None:
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def bench_lib():
    from paper_2511_07035_amd import BENCH_LIB_PATH
    if not os.path.exists(BENCH_LIB_PATH):
        raise ImportError(f"{BENCH_LIB_PATH} missing: python -m paper_2511_07035_amd.build")
    L = ctypes.CDLL(BENCH_LIB_PATH)
    L.gockpt_bench_spin.argtypes = [ctypes.c_void_p, ctypes.c_double, ctypes.c_int]
    L.gockpt_bench_spin.restype = ctypes.c_int
    L.gockpt_bench_copy.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_uint64, ctypes.c_int,
                                    ctypes.c_void_p]
    L.gockpt_bench_copy.restype = ctypes.c_int
    L.gockpt_bench_wallclock_khz.restype = ctypes.c_int
    L.gockpt_bench_stream.argtypes = [ctypes.c_int] + [ctypes.c_void_p] * 5 + [ctypes.c_uint64, ctypes.c_void_p]
    L.gockpt_bench_stream.restype = ctypes.c_int
    L.gockpt_bench_hog.argtypes = [ctypes.c_void_p, ctypes.c_double, ctypes.c_int]
    L.gockpt_bench_hog.restype = ctypes.c_int
    L.gockpt_bench_divsqrt.argtypes = [ctypes.c_void_p] * 4 + [ctypes.c_uint64, ctypes.c_void_p]
    L.gockpt_bench_convert.argtypes = [ctypes.c_int, ctypes.c_uint64, ctypes.c_uint64, ctypes.c_void_p, ctypes.c_void_p]
    L.gockpt_bench_convert.restype = ctypes.c_int
    L.gockpt_bench_divsqrt.restype = ctypes.c_int
    return L


# Sources of the fused kernel: a committed counter summary belongs to them
# only while their hash is the one it records.
TRAFFIC_SOURCES = ["paper_2511_07035_amd/csrc/gockpt_kernels.hip", "paper_2511_07035_amd/csrc/gockpt_contract.h",
                   "paper_2511_07035_amd/csrc/gockpt_internal.h"]
# The counter runs a traffic summary comes from (rocprofv3 pass per counter).
COUNTER_ARGS = ("--warmup 0 --steps {K} --stall-windows 0 --no-cpu-baseline --no-verify --no-schemes --tfb-ms 1 "
                "--copy-mib 256 --persist none")
COUNTER_CMD = ("rocprofv3 --pmc {ctr} --output-format csv -d {dir}/pmc_{tag}_{wl} -o {tag} -- "
               "python3 -u bench.py --workload {wl} " + COUNTER_ARGS)


def traffic_path(workload: str, out_dir: str | None = None) -> str:
    return os.path.join(out_dir or os.path.join(ROOT, "profiles"), f"fused_kernel_{workload}_traffic.json")


def kernel_sources_sha() -> str:
    import hashlib
    h = hashlib.sha256()
    for f in TRAFFIC_SOURCES:
        with open(os.path.join(ROOT, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def measured_traffic(workload: str, steps, out_dir: str | None = None):
    """HBM bytes per launch of the fused kernel over the window steps `steps`
    (their numbers s, one per timed launch), from the committed counter
    summary of this workload (FETCH_SIZE and WRITE_SIZE per window step,
    calibrated on a copy kernel of known size); None without a summary, or
    when the kernel sources have changed since the counters were taken."""
    path = traffic_path(workload, out_dir)
    if not os.path.exists(path) or not steps:
        return None
    t = json.load(open(path))
    if t.get("workload") != workload or t.get("source_sha256") != kernel_sources_sha():
        return None
    per = {int(w["s"]): float(w["traffic_bytes"]) for w in t["window_steps"]}
    if any(int(x) not in per for x in steps):
        return None
    return round(sum(per[int(x)] for x in steps) / len(steps))


def summarize_traffic(fetch_csv: str, write_csv: str, bench_json: str, out_dir: str | None = None) -> None:
    """profiles/fused_kernel_<workload>_traffic.{json,md} from the two counter
    runs: every fused_kernel dispatch is matched, in order, with the window
    step the bench ran it for (0: a plain step), the copy probe's 4 GiB copy
    kernel calibrates both counters, and each window step's traffic is set
    beside its algorithmic bytes."""
    import csv
    line = [ln for ln in open(bench_json) if ln.startswith("{")][-1]
    b = json.loads(line)
    # the runs' output directory (the one holding pmc_fetch_<workload>/), as
    # the commands named it: relative to the repository root when inside it
    run_dir = os.path.dirname(os.path.dirname(os.path.abspath(fetch_csv)))
    if run_dir.startswith(ROOT + os.sep):
        run_dir = os.path.relpath(run_dir, ROOT)
    wl, n, K = b["config"]["workload"], b["config"]["n_elems"], b["config"]["K"]
    order = b["fused_dispatch_steps"]
    alg = {int(k): int(v) for k, v in b["window_alg_bytes"].items()}

    def rows(path):
        out = {"fused": [], "copy": [], "prepass": []}
        for r in csv.DictReader(open(path)):
            k = r["Kernel_Name"]
            key = ("fused" if "gockpt::fused_kernel" in k else "copy" if "::copy_kernel(" in k
                   else "prepass" if "gockpt::prepass_kernel" in k else None)
            if key:
                out[key].append(float(r["Counter_Value"]))
        return out

    fe, wr = rows(fetch_csv), rows(write_csv)
    for name, r in (("FETCH_SIZE", fe), ("WRITE_SIZE", wr)):
        if len(r["fused"]) != len(order):
            raise SystemExit(f"{name}: {len(r['fused'])} fused_kernel dispatches, the bench ran {len(order)}")
    copy_kib = (4 << 30) / 1024
    f_fac = copy_kib / (sum(fe["copy"]) / len(fe["copy"]))
    w_fac = copy_kib / (sum(wr["copy"]) / len(wr["copy"]))
    per = {}
    for s_, f, w in zip(order, fe["fused"], wr["fused"]):
        per.setdefault(int(s_), []).append((f, w))
    steps = []
    for s_ in range(1, K + 1):
        fw = per.get(s_, [])
        if not fw:
            continue
        f = sum(x for x, _ in fw) / len(fw)
        w = sum(y for _, y in fw) / len(fw)
        steps.append({"s": s_, "FETCH_SIZE_KiB": f, "WRITE_SIZE_KiB": w, "traffic_bytes": (f * f_fac + w * w_fac) * 1024,
                      "algorithmic_bytes": alg.get(s_), "launches": len(fw)})
    plain = per.get(0, [])
    pre_t = [(f * f_fac + w * w_fac) * 1024 for f, w in zip(fe["prepass"], wr["prepass"])]
    t = {"kernel": "gockpt::fused_kernel", "workload": wl, "n": n, "K": K, "source_sha256": kernel_sources_sha(),
         "sources": TRAFFIC_SOURCES,
         "commands": [COUNTER_CMD.format(ctr=c, tag=g, wl=wl, K=K, dir=run_dir) for c, g in (("FETCH_SIZE", "fetch"),
                                                                                             ("WRITE_SIZE", "write"))],
         "calibration": {"copy_kernel_bytes_read": 4 << 30, "copy_kernel_bytes_written": 4 << 30,
                         "FETCH_SIZE_KiB": copy_kib / f_fac, "WRITE_SIZE_KiB": copy_kib / w_fac,
                         "fetch_factor": f_fac, "write_factor": w_fac},
         "window_steps": steps,
         "traffic_bytes_per_launch": sum(x["traffic_bytes"] for x in steps) / len(steps),
         "algorithmic_bytes_per_launch": sum(x["algorithmic_bytes"] for x in steps) / len(steps),
         "plain_step_traffic_bytes": (sum((f * f_fac + w * w_fac) * 1024 for f, w in plain) / len(plain)
                                      if plain else None),
         "plain_step_algorithmic_bytes": 28 * n,
         "prepass_traffic_bytes": sum(pre_t) / len(pre_t) if pre_t else None, "prepass_algorithmic_bytes": 2 * n}
    with open(traffic_path(wl, out_dir), "w") as fh:
        json.dump(t, fh, indent=1)
    md = traffic_path(wl, out_dir)[:-5] + ".md"
    c = t["calibration"]
    with open(md, "w") as f:
        f.write(f"# HBM traffic of the fused update+pack kernel -- {wl} (n = {n:,}, K = {K})\n\n")
        f.write("Two counter passes, each a run of its own (TMPDIR=/tmp, repository root), then the summary:\n\n")
        for cmd in t["commands"]:
            f.write(f"    {cmd}\n")
        f.write(f"    python3 bench.py --summarize-traffic <fetch counter_collection.csv> "
                f"<write counter_collection.csv> <the fetch run's stdout>\n\n")
        f.write("The bench's 4 GiB copy kernel (4 GiB read + 4 GiB written per dispatch) runs in the same process and "
                "calibrates the counters:\n\n")
        f.write("| counter | copy kernel (KiB/dispatch) | expected KiB | factor |\n|---|---|---|---|\n"
                f"| FETCH_SIZE | {c['FETCH_SIZE_KiB']:.0f} | {copy_kib:.0f} | {c['fetch_factor']:.5f} |\n"
                f"| WRITE_SIZE | {c['WRITE_SIZE_KiB']:.0f} | {copy_kib:.0f} | {c['write_factor']:.5f} |\n\n")
        f.write("Fused kernel per window step (traffic = FETCH x fetch factor + WRITE x write factor; algorithmic = "
                "28 B per element + the bytes the step packed into the ring):\n\n")
        f.write("| s | FETCH_SIZE KiB | WRITE_SIZE KiB | traffic bytes | algorithmic bytes | traffic / algorithmic |\n"
                "|---|---|---|---|---|---|\n")
        for x in steps:
            ratio = x["traffic_bytes"] / x["algorithmic_bytes"] if x["algorithmic_bytes"] else float("nan")
            f.write(f"| {x['s']} | {x['FETCH_SIZE_KiB']:.0f} | {x['WRITE_SIZE_KiB']:.0f} | {x['traffic_bytes']:.5g} | "
                    f"{x['algorithmic_bytes']:.5g} | {ratio:.5f} |\n")
        f.write(f"\nMean per launch: traffic {t['traffic_bytes_per_launch']:.5g} B, algorithmic "
                f"{t['algorithmic_bytes_per_launch']:.5g} B (ratio "
                f"{t['traffic_bytes_per_launch'] / t['algorithmic_bytes_per_launch']:.5f}).\n")
        if t["plain_step_traffic_bytes"]:
            f.write(f"Plain step (no pack): traffic {t['plain_step_traffic_bytes']:.5g} B vs 28 B x n = {28 * n:.5g} B.\n")
        if t["prepass_traffic_bytes"]:
            f.write(f"Prepass: traffic {t['prepass_traffic_bytes']:.5g} B vs 2 B x n = "
                    f"{2 * n:.5g} B.\n")
        f.write(f"\nKernel sources these counters belong to (sha256 over {', '.join(TRAFFIC_SOURCES)}): "
                f"`{t['source_sha256']}`.  bench.py reports `roofline.traffic` from the JSON beside this file, per "
                "timed window step, only while that hash matches.\n")
    print(f"wrote {traffic_path(wl, out_dir)} and {md}")


def fused_bytes(n: int, bounds, s: int) -> int:
    """Algorithmic HBM bytes of the fused update+pack at window step s when
    the whole pack goes through the ring and the step is applied."""
    return 28 * n + 12 * int(bounds[s] - bounds[s - 1]) + 2 * int(bounds[s - 1])


def fused_bytes_measured(n: int, ring_bytes: float, skipped: bool) -> int:
    """Algorithmic HBM bytes the fused kernel moved at one window step: the
    update (28 B per element) plus the pack stores into the ring; a skipped
    step only packs (reads and writes the packed bytes).  Bytes copied
    straight from the live buffers are the copy engine's, not the kernel's."""
    r = int(ring_bytes)
    return 2 * r if skipped else 28 * n + r


def d2h_bytes(bounds, s: int) -> int:
    return 12 * int(bounds[s] - bounds[s - 1]) + 2 * int(bounds[s - 1]) + RECORD_BYTES


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=8, help="timed window steps")
    ap.add_argument("--warmup", type=int, default=8, help="untimed window steps (whole windows)")
    import synth
    ap.add_argument("--workload", default="llama13b_k32", choices=sorted(synth.WORKLOADS))
    ap.add_argument("--tfb-ms", default="auto",
                    help="forward/backward stand-in per step in ms; auto = 6*N*8192 flop at 1 PFLOP/s")
    ap.add_argument("--ring-gib", type=float, default=None)
    ap.add_argument("--copy-mib", type=float, default=64)
    ap.add_argument("--threads", type=int, default=16, help="host restore threads")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=12.0)
    ap.add_argument("--no-verify", action="store_true")
    ap.add_argument("--no-probes", action="store_true")
    ap.add_argument("--pageable", choices=["auto", "yes", "no"], default="auto",
                    help="host arena in pageable memory through pinned staging (auto: if the window exceeds "
                         "--pin-limit-gib)")
    ap.add_argument("--pin-limit-gib", type=float, default=48.0)
    ap.add_argument("--staging-gib", type=float, default=32.0,
                    help="pinned staging for a pageable arena; holding a whole step's copies keeps the host from "
                         "waiting for slots")
    ap.add_argument("--copy-threads", type=int, default=16,
                    help="worker threads moving landed staging slots into a pageable arena")
    ap.add_argument("--replay-every", type=int, default=-1,
                    help="in-window replay every R steps (-1 auto: 0 unless the window's host arena exceeds "
                         "--host-limit-gib, then the largest R that fits)")
    ap.add_argument("--host-limit-gib", type=float, default=200.0)
    ap.add_argument("--no-schemes", dest="schemes", action="store_false",
                    help="skip the stall comparison of the checkpoint schemes")
    ap.add_argument("--scheme-reps", type=int, default=3)
    ap.add_argument("--schemes-pageable", action="store_true",
                    help="run the scheme comparison on a pageable-arena workload too (the lazy-policy schemes only: "
                         "Async-O, GoCkpt-O with and without the ring, Async-O into the ring)")
    ap.add_argument("--plan", action="store_true",
                    help="run the window planner's choice next to the configured window (predicted vs measured stall)")
    ap.add_argument("--plan-max-k", type=int, default=7)
    ap.add_argument("--plan-reps", type=int, default=2)
    ap.add_argument("--late-plan", choices=sorted(RING_PLANS), default="device",
                    help="ring plan of the windows: query (space freed when the host calls the step), host (the "
                         "calling thread waits until the device reaches the update), device (the whole ring, the "
                         "device waits for the copies of the reused ranges; never blocks the host)")
    ap.add_argument("--defer-copies", action="store_true",
                    help="windows queue each step's copies at the next library call (gockpt_window_opts."
                         "defer_copies) instead of in the step itself")
    ap.add_argument("--persist", default="auto",
                    help="directory to persist the restored checkpoint to and load it back from (auto: under "
                         "$TMPDIR when it has room; none: skip)")
    ap.add_argument("--stall-windows", type=int, default=3,
                    help="whole windows, each with the step after it and no host synchronisation inside, whose "
                         "checkpoint stall is measured; the median is reported")
    ap.add_argument("--flush-mall", choices=["auto", "yes", "no"], default="auto",
                    help="write 512 MiB before each update so the last-level cache holds none of the state "
                         "(auto: when the state is under 4 GiB)")
    ap.add_argument("--grad-dtype", choices=["bf16", "fp16"], default="bf16",
                    help="gradient format (the paper's FP16 or BF16)")
    ap.add_argument("--shard", default=None, metavar="I/P",
                    help="run rank I's share of a P-rank ZeRO-1 data-parallel split: the flat range "
                         "[I*N/P, (I+1)*N/P) at 256-element alignment with the tensor boundaries inside it; "
                         "T_fb stays the whole model's (every rank runs the whole forward/backward)")
    ap.add_argument("--no-overflow-check", action="store_true",
                    help="steps neither test the gradients for inf/NaN nor compute their norm, so no prepass runs "
                         "(bf16 training without loss scaling); not with dynamic loss scaling")
    ap.add_argument("--found-inf", action="store_true",
                    help="the skip decisions come from a caller-side found-inf flag (as a gradient scaler's, set "
                         "here at the workload's planted-inf steps) and no norm is computed, so no prepass runs")
    ap.add_argument("--bucket-scans", type=int, default=0, metavar="B",
                    help="the backward stand-in finishes the gradients in B buckets (last first) and each bucket's "
                         "overflow test and norm runs on a side stream as soon as it is written (gockpt_scan_grads), "
                         "beside the rest of the backward, instead of the prepass before the update")
    ap.add_argument("--fb", choices=["spin", "gemm", "launches"], default="spin",
                    help="forward/backward stand-in: a kernel waiting T_fb on one wavefront per compute unit "
                         "(spin), or bf16 8192^3 matrix products over every compute unit for about T_fb (gemm), "
                         "which also shows any slowdown the window's copies cause to compute, or --fb-kernels short "
                         "kernels launched one by one from Python (launches), as an eager training loop launches its "
                         "forward and backward: a library call that holds the calling thread then leaves the device "
                         "idle while the host catches up")
    ap.add_argument("--max-ahead", type=int, default=0,
                    help="the training loop keeps at most this many steps in flight: after each step it waits until "
                         "the device has finished the step that many steps back (as a loop that reads the loss each "
                         "step does); 0: no limit")
    ap.add_argument("--sync-loss", action="store_true",
                    help="the training loop waits for each step's forward before launching its backward, as a loop "
                         "that reads the loss every step does")
    ap.add_argument("--fb-kernels", type=int, default=8000,
                    help="kernels per step of the launches stand-in (a third of them in the forward)")
    ap.add_argument("--placement", choices=["slab", "packed"], default="slab",
                    help="HBM layout of the five state arrays (see StateSlab)")
    ap.add_argument("--summarize-traffic", nargs=3, metavar=("FETCH_CSV", "WRITE_CSV", "BENCH_JSON"),
                    help="write the committed traffic summary from two counter runs and exit")
    return ap.parse_args()


class GemmStandIn:
    """Forward/backward stand-in made of bf16 matrix products (torch's
    library GEMM) on the compute stream, as many as take about T_fb."""

    N = 8192

    def __init__(self, torch, stream, tfb_ms: float):
        self.torch, self.stream = torch, stream
        g = torch.Generator(device="cuda").manual_seed(1)
        self.a = torch.randn(self.N, self.N, device="cuda", dtype=torch.bfloat16, generator=g)
        self.b = torch.randn(self.N, self.N, device="cuda", dtype=torch.bfloat16, generator=g)
        self.c = torch.empty(self.N, self.N, device="cuda", dtype=torch.bfloat16)
        self._run(50)  # clocks up before the calibration
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        self._run(50)
        e1.record(stream)
        torch.cuda.synchronize()
        self.gemm_ms = e0.elapsed_time(e1) / 50
        total = max(3, round(tfb_ms / self.gemm_ms))
        self.n_fwd = total // 3
        self.n_bwd = total - self.n_fwd
        self.tflops = 2 * self.N ** 3 / (self.gemm_ms * 1e-3) / 1e12

    def _run(self, k: int) -> None:
        with self.torch.cuda.stream(self.stream):
            for _ in range(k):
                self.torch.matmul(self.a, self.b, out=self.c)

    def forward(self) -> None:
        self._run(self.n_fwd)

    def backward(self, parts: int = 1, i: int = 0) -> None:
        """The backward, or piece i of it cut into `parts` (the pieces add up
        to the whole)."""
        self._run(self.n_bwd * (i + 1) // parts - self.n_bwd * i // parts)

    def describe(self) -> dict:
        return {"gemm": f"bf16 {self.N}^3", "gemm_ms": round(self.gemm_ms, 4), "tflops": round(self.tflops, 1),
                "per_step": self.n_fwd + self.n_bwd, "fb_ms": round((self.n_fwd + self.n_bwd) * self.gemm_ms, 2)}


class LaunchStandIn:
    """Forward/backward stand-in launched as many short kernels, one host
    call each, like an eager training loop: T_fb is split evenly over
    n_kernels spin kernels (a third in the forward), each launched through
    ctypes on the compute stream."""

    def __init__(self, B, stream, tfb_ms: float, bwd_ms: float, n_kernels: int):
        self.B, self.stream = B, stream
        self.n_fwd = max(1, n_kernels // 3)
        self.n_bwd = max(1, n_kernels - self.n_fwd)
        self.fwd_each = tfb_ms / 3.0 / self.n_fwd
        self.bwd_total = bwd_ms

    def _run(self, k: int, each_ms: float) -> None:
        h = self.stream.cuda_stream
        spin = self.B.gockpt_bench_spin
        for _ in range(k):
            if spin(h, each_ms, 1) != 0:
                raise RuntimeError("spin launch failed")

    def forward(self) -> None:
        self._run(self.n_fwd, self.fwd_each)

    def backward(self, parts: int = 1, i: int = 0) -> None:
        k = self.n_bwd * (i + 1) // parts - self.n_bwd * i // parts
        if k > 0 and self.bwd_total > 0:
            self._run(k, self.bwd_total / self.n_bwd)

    def describe(self) -> dict:
        return {"launches": self.n_fwd + self.n_bwd, "forward_kernel_ms": round(self.fwd_each, 5),
                "backward_kernel_ms": round(self.bwd_total / self.n_bwd, 5)}


def link_probe(torch, stream, reps: int = 20) -> float:
    n = 1 << 30
    d = torch.empty(n, dtype=torch.uint8, device="cuda")
    d.fill_(7)
    h = torch.empty(n, dtype=torch.uint8, pin_memory=True)
    res = []
    for _ in range(reps):
        torch.cuda.synchronize()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        with torch.cuda.stream(stream):
            h.copy_(d, non_blocking=True)
        e1.record(stream)
        torch.cuda.synchronize()
        res.append(n / (e0.elapsed_time(e1) * 1e-3) / 1e9)
    del d, h
    return statistics.median(res)


def engine_probe(torch, B, copy_stream, hog_ms: float = 100.0) -> dict:
    """Do the device-to-host copies need compute units?  A kernel holds every
    wave slot (8 blocks of 4 waves per compute unit) for hog_ms while 512 MiB
    go to pinned memory on the copy stream.  Copies on the DMA engines finish
    beside it at the link rate; copies run as kernels would wait for it."""
    n = 512 << 20
    d = torch.empty(n, dtype=torch.uint8, device="cuda")
    d.fill_(5)
    h = torch.zeros(n, dtype=torch.uint8, pin_memory=True)
    hog_stream = torch.cuda.Stream()
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    h.copy_(d)  # first touch of the pinned pages by the device, outside the measurement
    torch.cuda.synchronize()
    h.zero_()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
    ev[0].record(hog_stream)
    rc = B.gockpt_bench_hog(hog_stream.cuda_stream, hog_ms, 8 * cus)
    assert rc == 0, rc
    ev[1].record(hog_stream)
    time.sleep(0.01)  # the hog is resident before the copies are queued
    ev[2].record(copy_stream)
    with torch.cuda.stream(copy_stream):
        for a in range(0, n, 64 << 20):  # the library's default copy size
            h[a:a + (64 << 20)].copy_(d[a:a + (64 << 20)], non_blocking=True)
    ev[3].record(copy_stream)
    torch.cuda.synchronize()
    ok = bool((h[::1 << 16] == 5).all())
    out = {"hog_ms": round(ev[0].elapsed_time(ev[1]), 2), "copy_ms": round(ev[2].elapsed_time(ev[3]), 2),
           "copy_end_ms": round(ev[0].elapsed_time(ev[3]), 2), "copied": ok}
    out["copy_gbs"] = round(n / (out["copy_ms"] * 1e-3) / 1e9, 1)
    out["copies_beside_full_occupancy"] = out["copy_end_ms"] < out["hog_ms"]
    del d, h
    return out


def copy_probe(torch, B, reps: int = 10) -> float:
    """Plain 16-byte device copy of 4 GiB: achievable read+write GB/s."""
    nbytes = 4 << 30
    a = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    b = torch.empty_like(a)
    a.fill_(1)
    res = []
    s = torch.cuda.current_stream()
    for _ in range(reps):
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(s)
        rc = B.gockpt_bench_copy(b.data_ptr(), a.data_ptr(), nbytes, 256 * 32, s.cuda_stream)
        assert rc == 0, rc
        e1.record(s)
        torch.cuda.synchronize()
        res.append(2 * nbytes / (e0.elapsed_time(e1) * 1e-3) / 1e9)
    del a, b
    return statistics.median(res)


def stream_probe(torch, B, grad, master, exp_avg, exp_avg_sq, weight, reps: int = 5) -> dict:
    """HBM ceilings on the workload's own buffers (run before they are
    initialised): read-only, write-only and the fused-update memory twin."""
    n = master.numel() // 4 * 4
    s = torch.cuda.current_stream()

    def best(launch, nbytes):
        out = []
        for i in range(reps + 1):
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record(s)
            rc = launch()
            assert rc == 0, rc
            e1.record(s)
            torch.cuda.synchronize()
            if i:
                out.append(nbytes / (e0.elapsed_time(e1) * 1e-3) / 1e9)
        return round(max(out), 1)

    nb = 4 * n
    return {
        "read_gbs": best(lambda: B.gockpt_bench_stream(0, master.data_ptr(), None, None, None, None, nb,
                                                       s.cuda_stream), nb),
        "write_gbs": best(lambda: B.gockpt_bench_stream(1, exp_avg.data_ptr(), None, None, None, None, nb,
                                                        s.cuda_stream), nb),
        "update_twin_gbs": best(lambda: B.gockpt_bench_stream(2, grad.data_ptr(), master.data_ptr(),
                                                              exp_avg.data_ptr(), exp_avg_sq.data_ptr(),
                                                              weight.data_ptr(), n, s.cuda_stream), 28 * n),
    }


SCHEMES = {
    # name: (window length, wait policy, ring used).  K = 1: one snapshot of
    # the whole state; the GoCkpt schemes spread it over the window's K steps.
    "async": ("1", 2, False),          # blocking copy of the whole state
    "async_o": ("1", 0, False),        # the copy overlaps one step; the next update waits
    "gockpt": ("K", 1, False),         # parts over K steps, explicit wait for the gradients
    "gockpt_o": ("K", 0, False),       # gradient copies hidden behind the next forward
    "gockpt_o_ring": ("K", 0, True),   # this library's default: pack into the HBM ring
    "async_o_ring": ("1", 0, True),    # whole-state snapshot into the HBM ring
}


def persist_roundtrip(torch, sess, n, args):
    """Persist the checkpoint the last restore left in the arena (parallel
    piece writes, fdatasync, metadata last), then load it back into the
    device state, which must not change.  Reading hits the page cache the
    write just filled."""
    import shutil
    import tempfile
    need = 12 * n
    if args.persist == "auto":
        base = os.environ.get("TMPDIR", tempfile.gettempdir())
        if shutil.disk_usage(base).free < 2 * need + (8 << 30):
            log(f"persist: skipped, {base} lacks room for {need / 1e9:.1f} GB")
            return None
        root = tempfile.mkdtemp(prefix="gockpt_bench_", dir=base)
    else:
        root = args.persist
        os.makedirs(root, exist_ok=True)
    d = os.path.join(root, "ckpt")
    try:
        before = [t.clone() for t in (sess.master[:1 << 20], sess.exp_avg_sq[-(1 << 20):])]
        sess.persist(d, user_meta="bench\n", nthreads=args.threads)
        st = sess.persist_wait()
        t0 = time.perf_counter()
        info = sess.load(d, nthreads=args.threads)
        load_ms = (time.perf_counter() - t0) * 1e3
        same = all(bool(torch.equal(a, b)) for a, b in
                   zip(before, (sess.master[:1 << 20], sess.exp_avg_sq[-(1 << 20):])))
        out = {"bytes": int(st.bytes), "write_ms": round(st.ms, 1), "write_gbs": round(st.bytes / st.ms / 1e6, 2),
               "load_ms": round(load_ms, 1), "load_gbs": round(st.bytes / load_ms / 1e6, 2),
               "load_from": "page cache", "threads": args.threads, "t": int(info.t),
               "device_state_unchanged": same}
        log(f"persist {st.bytes / 1e9:.1f} GB in {st.ms:.0f} ms ({out['write_gbs']} GB/s, synced); load "
            f"{load_ms:.0f} ms ({out['load_gbs']} GB/s incl. H2D); unchanged: {same}")
        return out
    finally:
        if args.persist == "auto":
            shutil.rmtree(root, ignore_errors=True)
        else:
            shutil.rmtree(d, ignore_errors=True)


class SpanTimer:
    """Compute-stream time of a span of training steps, with a window opened
    at its first step or without one; the stall of a window is the span with
    it minus the span without it, median over reps after one warm-up pair."""

    def __init__(self, torch, sess, train_step, threads: int, pageable: bool, replay_every: int = 0):
        self.torch, self.sess, self.train_step = torch, sess, train_step
        self.threads, self.pageable, self.replay_every = threads, pageable, replay_every
        self.gstep = 10_000_000

    def span(self, steps: int, window: dict | None = None) -> float:
        torch, sess = self.torch, self.sess
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record(sess.compute)
        if window is not None:
            kw = len(window["bounds"]) - 1  # in-window replay keeps a long window's host arena bounded
            sess.begin_window(window["bounds"], wait_policy=window.get("wait_policy", 0),
                              ring_off=window.get("ring_off", False), late_plan=window.get("late_plan", 0),
                              pageable=self.pageable, replay_threads=self.threads,
                              replay_every=self.replay_every if 0 < self.replay_every < kw else 0, timing=False)
        for _ in range(steps):
            self.gstep += 1
            self.train_step(0, self.gstep)  # no planted infs: every span does the same updates
        e1.record(sess.compute)
        torch.cuda.synchronize()
        if window is not None:
            sess.drain(blocking=True)
            sess.restore(nthreads=self.threads)
        return e0.elapsed_time(e1)

    def stall(self, window: dict, steps: int, reps: int) -> float:
        out = []
        for _ in range(reps + 1):
            ref = self.span(steps)
            out.append(self.span(steps, window) - ref)
        return statistics.median(out[1:])


def model_params(n, tfb_ms, plain_ms, upd_ms, pack_bytes, fused_gbs, link_gbs):
    """Inputs of the library's window model from this run's measurements:
    forward = a third of T_fb (the stand-in's split), update without pack =
    28 B per element at the fused kernel's rate, backward = the rest of a
    plain step (backward stand-in, gradient writes, prepass)."""
    t_fwd = tfb_ms / 3.0
    t_upd = upd_ms * (28.0 * n) / (28.0 * n + pack_bytes)
    return dict(t_fwd_ms=t_fwd, t_bwd_ms=max(0.0, plain_ms - t_fwd - t_upd), t_upd_ms=t_upd,
                pack_gbs=fused_gbs, link_gbs=link_gbs)


def compare_schemes(timer, bounds, K, n, plain_ms, link_gbs, tfb_ms, model, ring_bytes, copy_bytes, args):
    """Checkpoint stall of each scheme on the same steps (a span of K + 2
    steps), the library's window model's prediction beside it, and the closed
    forms of the paper's Sec. 4.2.3 with the measured host link."""
    from paper_2511_07035_amd import gockpt_simulate_window
    span = K + 2
    res = {}
    for name, (kind, pol, ring) in SCHEMES.items():
        if args.schemes_pageable and pol != 0:
            continue  # a pageable arena takes the lazy policy only
        b = [0, n] if kind == "1" else bounds
        st = timer.stall(dict(bounds=b, wait_policy=pol, ring_off=not ring, late_plan=RING_PLANS[args.late_plan]),
                         span, args.scheme_reps)
        entry = {"stall_ms_per_checkpoint": round(st, 2), "stall_ms_per_step": round(st / span, 3),
                 "window_steps": len(b) - 1}
        if model is not None:
            pred, _ = gockpt_simulate_window(b, n, model["t_fwd_ms"], model["t_bwd_ms"], model["t_upd_ms"],
                                             model["link_gbs"], pack_gbs=model["pack_gbs"], wait_policy=pol,
                                             ring_bytes=ring_bytes if ring else 0, copy_bytes=copy_bytes,
                                             ring_plan=model["ring_plan"], staging_bytes=model["staging_bytes"],
                                             host_gbs=model["host_gbs"])
            entry["predicted_ms"] = round(pred.stall_ms, 2)
        res[name] = entry
        log(f"scheme {name}: stall {st:.1f} ms per checkpoint"
            + (f" (model {entry['predicted_ms']:.1f})" if "predicted_ms" in entry else ""))
    if link_gbs:
        t_step = plain_ms if plain_ms else tfb_ms
        t_x = 12 * n / (link_gbs * 1e9) * 1e3
        grads = sum(2 * int(bounds[s - 1]) for s in range(2, K + 1)) / (link_gbs * 1e9) * 1e3
        res["closed_forms"] = {"t_step_ms": round(t_step, 2), "state_copy_ms": round(t_x, 1),
                               "async_ms": round(t_x, 1), "async_o_ms": round(max(0.0, t_x - t_step), 1),
                               "gockpt_ms": round(grads, 1), "link_gbs": round(link_gbs, 2)}
    return res


def compare_plan(timer, bounds, K, n, model, ring_bytes, copy_bytes, tensor_ends, args):
    """The configured window against the window planner's choice (cap
    args.plan_max_k): predicted and measured checkpoint stall of each."""
    from paper_2511_07035_amd import gockpt_plan_window, gockpt_simulate_window
    common = dict(pack_gbs=model["pack_gbs"], ring_bytes=ring_bytes, copy_bytes=copy_bytes,
                  ring_plan=model["ring_plan"], staging_bytes=model["staging_bytes"], host_gbs=model["host_gbs"])
    args_m = (n, model["t_fwd_ms"], model["t_bwd_ms"], model["t_upd_ms"], model["link_gbs"])
    cfg_pred, _ = gockpt_simulate_window(bounds, *args_m, **common)
    pb, plan = gockpt_plan_window(*args_m, tensor_ends=tensor_ends, max_K=args.plan_max_k, **common)
    log(f"planner: K={plan.K}, predicted stall {plan.stall_ms:.1f} ms (configured K={K}: {cfg_pred.stall_ms:.1f} ms)")
    out = {"model": {k: round(v, 3) for k, v in model.items()}, "max_K": args.plan_max_k}
    for name, b in (("configured", bounds), ("planned", pb)):
        k = len(b) - 1
        st = timer.stall(dict(bounds=b, late_plan=RING_PLANS[args.late_plan]), k + 2, args.plan_reps)
        pred = cfg_pred if name == "configured" else plan
        out[name] = {"K": k, "bounds": [int(x) for x in b], "predicted_stall_ms": round(pred.stall_ms, 2),
                     "measured_stall_ms": round(st, 2), "predicted_d2h_bytes": int(pred.d2h_bytes),
                     "predicted_spilled_bytes": int(pred.spilled_bytes)}
        log(f"{name} window K={k}: stall {st:.1f} ms measured, {pred.stall_ms:.1f} ms predicted")
    return out


def cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(wl, bounds_full, n_full: int, seed: int, target_s: float, threads: int, grad_dtype: str = "bf16"):
    """The oracle as it stands on the first n_s elements of the same workload:
    all K window steps (update + capture of what is sent) on one thread; the
    same work split over `threads` element ranges run concurrently (the C
    oracle releases the interpreter lock); and the oracle's replay-restore of
    the one-thread capture."""
    import concurrent.futures

    import oracle
    import synth

    K = wl["K"]
    dyn = wl["dynamic"]
    cfg = oracle.AdamWConfig(dynamic_scale=dyn, init_scale=65536.0 if dyn else 1.0, grad_dtype=grad_dtype)
    n_c = 1 << 18
    st = oracle.State(synth.master_cpu(n_c, seed))
    g = synth.grads_cpu(n_c, seed, 1, dtype=grad_dtype)
    t0 = time.perf_counter()
    oracle.adamw_step(st, g, cfg)
    per_elem_step = (time.perf_counter() - t0) / n_c
    n_s = int(target_s / max(per_elem_step * K, 1e-12))
    n_s = max(1 << 20, min(n_s, 1 << 26, n_full)) // 256 * 256
    frac = np.asarray(bounds_full, dtype=np.float64) / float(n_full)

    def scaled(n_part):
        b = (frac * n_part).astype(np.int64) // 8 * 8
        b[0], b[-1] = 0, n_part
        return b

    b = scaled(n_s)
    sched = synth.DYNSCALE_SCHEDULE if dyn else {}
    grads = np.stack([synth.grads_cpu(n_s, seed, s, law=wl["grad"], scale=sched.get(s, 1.0),
                                      plant_inf=s in wl["inf_steps"], dtype=grad_dtype) for s in range(1, K + 1)])
    p0 = synth.master_cpu(n_s, seed)
    st = oracle.State(p0, scale=cfg.init_scale)
    t0 = time.perf_counter()
    cap = oracle.window_capture(st, grads, b, cfg)
    dt = time.perf_counter() - t0
    nbytes = sum(fused_bytes(n_s, b, s) for s in range(1, K + 1))
    t0 = time.perf_counter()
    oracle.replay_restore(cap, cfg)
    dt_restore = time.perf_counter() - t0
    updates = sum((K - j) * int(b[j] - b[j - 1]) for j in range(1, K + 1))
    # the same sample on `threads` element ranges; the skip flags are global
    nonfinite = [int(oracle.any_nonfinite(grads[s], grad_dtype)) for s in range(K)]
    edges = np.linspace(0, n_s, threads + 1).astype(np.int64) // 256 * 256
    edges[-1] = n_s
    jobs = []
    for lo, hi in zip(edges[:-1], edges[1:]):
        if hi > lo:
            jobs.append((oracle.State(p0[lo:hi], scale=cfg.init_scale), np.ascontiguousarray(grads[:, lo:hi]),
                         scaled(int(hi - lo))))
    t0 = time.perf_counter()
    with concurrent.futures.ThreadPoolExecutor(len(jobs)) as ex:
        list(ex.map(lambda j: oracle.window_capture(j[0], j[1], j[2], cfg, nonfinite=nonfinite), jobs))
    dt_par = time.perf_counter() - t0
    return {"value": round(nbytes / dt / 1e9, 3), "unit": "GB/s", "cores": 1, "kind": "oracle",
            "sample": f"first {n_s} elements of the {n_full}-element flat space, all {K} window steps "
                      f"(update + capture of the sent part and gradients), part bounds scaled from the full ones",
            "seconds": round(dt, 3), "elements_per_s": round(n_s * K / dt, 1),
            "parallel": {"value": round(nbytes / dt_par / 1e9, 3), "unit": "GB/s", "cores": len(jobs),
                         "seconds": round(dt_par, 3), "note": "the same sample split into element ranges"},
            "replay_restore": {"element_updates": updates, "seconds": round(dt_restore, 3),
                               "updates_per_s": round(updates / dt_restore, 1), "cores": 1},
            "cpu_model": cpu_model()}


def host_cores() -> int:
    """Host threads the oracle's parallel leg may use: the cores this process
    may run on, at most 16 (a GPU's share of the host)."""
    try:
        c = len(os.sched_getaffinity(0))
    except (AttributeError, OSError):
        c = os.cpu_count() or 1
    return max(1, min(16, c))


def main():
    args = parse()
    if args.summarize_traffic:
        summarize_traffic(*args.summarize_traffic)
        return
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (--gpus {args.gpus} asked); the single-GPU path is the per-rank "
              f"kernel of a data-parallel run and no multi-GPU figure is produced.", file=sys.stderr)
        sys.exit(2)
    if args.steps < 1:
        sys.exit("--steps must be >= 1")
    import torch

    import synth
    from paper_2511_07035_amd import GOCKPT_ALIGN_ELEMS, Session, gockpt_plan_bounds

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    B = bench_lib()
    wl = synth.WORKLOADS[args.workload]
    if args.no_overflow_check and wl["dynamic"]:
        sys.exit("--no-overflow-check: dynamic loss scaling needs the overflow test")
    if sum([args.no_overflow_check, args.found_inf, args.bucket_scans > 0]) > 1:
        sys.exit("--found-inf, --no-overflow-check and --bucket-scans exclude each other")
    no_prepass = args.no_overflow_check or args.found_inf or args.bucket_scans > 0
    no_norm = args.no_overflow_check or args.found_inf
    layout = synth.LAYOUTS[wl["layout"]]()
    n_model = synth.numel(layout)
    ends = synth.tensor_ends(layout)
    n, shard = n_model, None
    if args.shard:
        try:
            rank, P = (int(x) for x in args.shard.split("/"))
        except ValueError:
            sys.exit(f"--shard {args.shard}: expected I/P")
        if not (P >= 1 and 0 <= rank < P):
            sys.exit(f"--shard {args.shard}: need 0 <= I < P")
        lo = n_model * rank // P // 256 * 256
        hi = n_model if rank == P - 1 else n_model * (rank + 1) // P // 256 * 256
        ends = np.clip(ends, lo, hi) - lo
        ends = np.unique(ends[ends > 0])
        n, shard = int(hi - lo), {"rank": rank, "ranks": P, "range": [int(lo), int(hi)], "n_model": n_model}
    K = wl["K"]
    if wl["partition"] == "tensors":
        bounds = gockpt_plan_bounds(K, n, ends)
    else:
        bounds = gockpt_plan_bounds(K, n, align=256 if wl["partition"] == "bytes" else GOCKPT_ALIGN_ELEMS)
    if args.ring_gib is not None:
        ring_bytes = int(args.ring_gib * (1 << 30)) // 256 * 256
    else:
        ring_bytes = wl["ring_bytes"]  # None: what HBM has left, sized after the state is allocated
    tfb_ms = 6.0 * n_model * 8192 / 1e15 * 1e3 if args.tfb_ms == "auto" else float(args.tfb_ms)
    from paper_2511_07035_amd import gockpt_arena_layout_ex
    R = args.replay_every
    if R < 0:
        R = 0
        if gockpt_arena_layout_ex(K, bounds, n, 0)[0].total > args.host_limit_gib * (1 << 30):
            R = K - 1
            while R > 1 and gockpt_arena_layout_ex(K, bounds, n, R)[0].total > args.host_limit_gib * (1 << 30):
                R -= 1
    arena_total = gockpt_arena_layout_ex(K, bounds, n, R)[0].total
    pageable = args.pageable == "yes" or (args.pageable == "auto" and arena_total > args.pin_limit_gib * (1 << 30))
    staging = int(args.staging_gib * (1 << 30)) if pageable else 0
    log(f"workload {args.workload}{' shard ' + args.shard if shard else ''}: n={n} K={K} ring={ring_bytes if ring_bytes is not None else 'auto'}, "
        f"T_fb={tfb_ms:.2f} ms, arena "
        f"{arena_total / 1e9:.1f} GB {'pageable via staging' if pageable else 'pinned'}, replay_every={R}")

    # ---- device state (inputs resident in HBM) --------------------------------
    from paper_2511_07035_amd import StateSlab
    # the staging ring comes out of the slab's gaps; keep room for the probes
    layout_state = StateSlab(n, placement=args.placement, reserve_bytes=24 << 30, grad_dtype=args.grad_dtype)
    master, exp_avg, exp_avg_sq = layout_state.master, layout_state.exp_avg, layout_state.exp_avg_sq
    grad, weight = layout_state.grad, layout_state.weight
    grad.zero_()
    log(f"state layout {args.placement}: array offsets (GiB) "
        f"{[round((t.data_ptr() - master.data_ptr()) / (1 << 30), 1) for t in (master, exp_avg, exp_avg_sq, grad, weight)]}")
    ring_t = None
    if ring_bytes is None:
        window = 12 * n + 2 * int(bounds[:-1].sum())
        room = max([g[1] for g in layout_state.gaps], default=0)
        room = max(room, torch.cuda.mem_get_info()[0] - (16 << 30))
        ring_bytes = max(0, min(room, window)) // 256 * 256
        log(f"ring {ring_bytes / (1 << 30):.1f} GiB (HBM left after the state)")
    if ring_bytes:
        ring_t = layout_state.take(ring_bytes)
    probe = None
    if not args.no_probes:
        probe = stream_probe(torch, B, grad, master, exp_avg, exp_avg_sq, weight)
        log(f"HBM probes on the workload buffers: {probe}")
    synth.master_dev_(master, args.seed)
    weight.copy_(master.to(torch.bfloat16))
    exp_avg.zero_()
    exp_avg_sq.zero_()
    sess = Session(n, master=master, exp_avg=exp_avg, exp_avg_sq=exp_avg_sq, weight=weight, grad=grad,
                   dynamic_scale=wl["dynamic"],
                   init_scale=65536.0 if wl["dynamic"] else 1.0, ring_bytes=ring_bytes,
                   copy_bytes=int(args.copy_mib * (1 << 20)) // 256 * 256, timing=True,
                   staging_bytes=staging, copy_threads=args.copy_threads, ring=ring_t, grad_dtype=args.grad_dtype,
                   check_overflow=not args.no_overflow_check, grad_norm=not no_norm,
                   found_inf=torch.zeros(1, dtype=torch.float32, device="cuda") if args.found_inf else None)
    torch.cuda.synchronize()
    sched = synth.DYNSCALE_SCHEDULE if wl["dynamic"] else {}

    flush_buf = None
    if args.flush_mall == "yes" or (args.flush_mall == "auto" and 16 * n < (4 << 30)):
        flush_buf = torch.empty(512 << 20, dtype=torch.uint8, device="cuda")

    fb = None
    if args.fb == "gemm" and tfb_ms > 0:
        fb = GemmStandIn(torch, sess.compute, tfb_ms)
        log(f"forward/backward stand-in: {fb.describe()}")

    scan_stream, scan_edges = None, None
    scan_tail = {}  # gstep -> events around the last bucket's scan, which runs on the compute stream
    host_in_lib = [0.0]  # host seconds inside gockpt_backward_begin and gockpt_step of the counted steps
    dispatch_steps = []  # window step (0: plain) of every fused-kernel launch, in order
    in_flight = []  # --max-ahead: events after the steps still in flight
    if args.bucket_scans > 0:
        scan_stream = torch.cuda.Stream()
        scan_edges = np.unique(np.append(np.linspace(0, n, args.bucket_scans + 1).astype(np.int64) // 256 * 256, n))

    # The gradient generation stands in for the backward's writes of the
    # gradients; it runs inside the backward's share of T_fb, so the backward
    # stand-in is shortened by its measured time and a step stays T_fb plus
    # the optimizer step.
    gen_ms = 0.0
    if tfb_ms > 0:
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        with torch.cuda.stream(sess.compute):
            synth.grads_dev_(sess.grad, args.seed, 1 << 40, law=wl["grad"])
            ev[0].record(sess.compute)
            for r in range(3):
                synth.grads_dev_(sess.grad, args.seed, (1 << 40) + r + 1, law=wl["grad"])
            ev[1].record(sess.compute)
        torch.cuda.synchronize()
        gen_ms = ev[0].elapsed_time(ev[1]) / 3
        log(f"gradient generation {gen_ms:.2f} ms per step (taken out of the backward stand-in)")
    bwd_ms = max(0.0, tfb_ms * 2.0 / 3.0 - gen_ms)
    if args.fb == "launches" and tfb_ms > 0:
        fb = LaunchStandIn(B, sess.compute, tfb_ms, bwd_ms, args.fb_kernels)
        log(f"forward/backward stand-in: {fb.describe()}")

    def train_step(s_in_window: int, gstep: int, spin: bool = True, count: bool = False):
        # forward (a third of T_fb), then the backward, which overwrites the
        # gradient buffer: gockpt_backward_begin sits between the two.
        # count: add the host time inside the library to host_in_lib.
        if spin and tfb_ms > 0:
            if fb is not None:
                fb.forward()
            else:
                rc = B.gockpt_bench_spin(sess.compute.cuda_stream, tfb_ms / 3.0, 256)
                assert rc == 0, rc
        if args.sync_loss:  # the loop reads the loss: it waits for the forward
            sess.compute.synchronize()
        h0 = time.perf_counter()
        sess.backward_begin()
        if count:
            host_in_lib[0] += time.perf_counter() - h0
        scale = sched.get(s_in_window, 1.0) if wl["dynamic"] else 1.0
        if scan_stream is not None:
            # the backward finishes the gradients bucket by bucket, last
            # first; each bucket is scanned beside the rest of the backward
            nb = len(scan_edges) - 1
            for j in reversed(range(nb)):
                a, b = int(scan_edges[j]), int(scan_edges[j + 1])
                if spin and tfb_ms > 0:
                    if fb is not None:
                        fb.backward(nb, nb - 1 - j)
                    elif bwd_ms > 0:
                        rc = B.gockpt_bench_spin(sess.compute.cuda_stream, bwd_ms / nb, 256)
                        assert rc == 0, rc
                with torch.cuda.stream(sess.compute):
                    synth.grads_dev_(sess.grad[a:b], args.seed, gstep * 4096 + j, law=wl["grad"], scale=scale,
                                     plant_inf=s_in_window in wl["inf_steps"] and j == nb - 1)
                if j > 0:
                    scan_stream.wait_stream(sess.compute)
                    sess.scan_grads(a, b, stream=scan_stream)
                elif s_in_window > 0:  # the last bucket: on the compute stream, no cross-stream hop
                    ea, eb = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                    ea.record(sess.compute)
                    sess.scan_grads(a, b)
                    eb.record(sess.compute)
                    scan_tail[gstep] = (ea, eb)
                else:
                    sess.scan_grads(a, b)
        else:
            if spin and tfb_ms > 0:
                if fb is not None:
                    fb.backward()
                elif bwd_ms > 0:
                    rc = B.gockpt_bench_spin(sess.compute.cuda_stream, bwd_ms, 256)
                    assert rc == 0, rc
            with torch.cuda.stream(sess.compute):
                synth.grads_dev_(sess.grad, args.seed, gstep, law=wl["grad"], scale=scale,
                                 plant_inf=s_in_window in wl["inf_steps"])
        if sess.found_inf is not None:  # the caller's overflow decision for this step
            with torch.cuda.stream(sess.compute):
                sess.found_inf.fill_(1.0 if s_in_window in wl["inf_steps"] else 0.0)
        if flush_buf is not None:  # evict the state from the 256 MB last-level cache
            rc = B.gockpt_bench_stream(1, flush_buf.data_ptr(), None, None, None, None, flush_buf.numel(),
                                       sess.compute.cuda_stream)
            assert rc == 0, rc
        h0 = time.perf_counter()
        sess.step(1e-4)
        if count:
            host_in_lib[0] += time.perf_counter() - h0
        dispatch_steps.append(s_in_window)
        if args.max_ahead > 0:  # the loop's own wait (outside the library)
            ev = torch.cuda.Event()
            ev.record(sess.compute)
            in_flight.append(ev)
            while len(in_flight) > args.max_ahead:
                in_flight.pop(0).synchronize()

    link_gbs = copy_gbs = engine = None
    if not args.no_probes:
        engine = engine_probe(torch, B, sess.copy)
        log(f"D2H beside a kernel holding every wave slot: {engine}")
        link_gbs = link_probe(torch, sess.copy)
        log(f"host link D2H {link_gbs:.1f} GB/s (1 GiB pinned, median of 20)")
        copy_gbs = copy_probe(torch, B)
        log(f"device copy kernel {copy_gbs:.0f} GB/s (read + write, 4 GiB)")

    gstep = 0

    plan_mode = RING_PLANS[args.late_plan]

    def run_window(n_timed: int | None, record: list, post: int = 0):
        """One K-step window; the first n_timed steps are inside the timed
        region (None: untimed), with a host synchronisation after the last
        of them.  post: plain steps run after the window's last step, before
        the drain, with no host synchronisation anywhere from the window's
        start to their end.  Returns the wall ms of the timed part, the
        restore meta, the window stats and the compute-stream ms from the
        window's start to the end of the post steps (None without them)."""
        nonlocal gstep
        # only the timed windows record the library's timing events: the
        # others (warm-up, stall) run as an untimed training loop would
        sess.begin_window(bounds, replay_every=R, pageable=pageable, replay_threads=args.threads,
                          late_plan=plan_mode, timing=n_timed is not None, defer_copies=args.defer_copies)
        torch.cuda.synchronize()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e2 = torch.cuda.Event(enable_timing=True)
        e0.record(sess.compute)
        t0 = time.perf_counter()
        wall = 0.0
        gsteps = []
        for s in range(1, K + 1):
            gstep += 1
            gsteps.append(gstep)
            timed = n_timed is not None and s <= n_timed
            train_step(s, gstep, count=timed)
            if n_timed is not None and s == n_timed:
                e1.record(sess.compute)
                torch.cuda.synchronize()
                wall = (time.perf_counter() - t0) * 1e3
        for _ in range(post):
            gstep += 1
            train_step(0, gstep)
        if post:
            e2.record(sess.compute)
        st = sess.drain(blocking=True)
        torch.cuda.synchronize()
        skips = sess.records()["skip"].astype(bool)
        if n_timed is not None:
            times = sess.step_times()
            # the last bucket's scan sits on the compute stream just before the
            # step: it belongs to the step's critical path
            tail = sum(scan_tail[g][0].elapsed_time(scan_tail[g][1]) for g in gsteps[:n_timed] if g in scan_tail)
            record.append((n_timed, times[:n_timed].copy(), st, e0.elapsed_time(e1), skips[:n_timed].copy(), tail))
        for g in gsteps:
            scan_tail.pop(g, None)
        meta = sess.restore(nthreads=args.threads)
        return wall, meta, st, (e0.elapsed_time(e2) if post else None)

    # ---- warmup: whole windows, drained and restored -----------------------------
    restore_ms = restore_updates = None
    for w in range(max(0, (args.warmup + K - 1) // K)):
        _, meta, st, _ = run_window(None, [])
        restore_ms, restore_updates = meta.restore_ms, meta.element_updates
        log(f"warmup window {w + 1}: restore {restore_ms:.0f} ms ({restore_updates} element updates, "
            f"{args.threads} threads); copies {st.bytes_d2h / 1e9:.2f} GB, spilled {st.bytes_spilled / 1e9:.2f} GB")

    # ---- the same steps without a window (stall reference) ------------------------
    plain_ms = host_plain_ms = None
    if tfb_ms > 0:
        torch.cuda.synchronize()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(sess.compute)
        n_plain = min(K, 8)
        host_in_lib[0] = 0.0
        for _ in range(n_plain):
            gstep += 1
            train_step(0, gstep, count=True)
        host_plain_ms = host_in_lib[0] * 1e3 / n_plain
        e1.record(sess.compute)
        torch.cuda.synchronize()
        plain_ms = e0.elapsed_time(e1) / n_plain
        log(f"plain steps (no window): {plain_ms:.2f} ms/step on the compute stream")

    # ---- timed: exactly args.steps window steps -----------------------------------
    recorded = []
    wall_ms = 0.0
    left = args.steps
    last_meta = None
    host_in_lib[0] = 0.0
    while left > 0:
        take = min(K, left)
        w_ms, last_meta, _, _ = run_window(take, recorded)
        wall_ms += w_ms
        left -= take
        log(f"timed window: {take} steps in {w_ms:.1f} ms")
    host_window_ms = host_in_lib[0] * 1e3 / args.steps  # only the timed steps were counted
    if last_meta is not None:
        restore_ms, restore_updates = last_meta.restore_ms, last_meta.element_updates
    ms_per_step = wall_ms / args.steps

    # ---- checks: the last timed window's restored checkpoint is the device state
    # after its step K (before the stall windows move the state on) ---------------
    verified = None
    if not args.no_verify:
        ap_, am_, av_ = sess.arena_state()
        ok = True
        chunk = 1 << 28
        for dev, host in ((sess.master, ap_), (sess.exp_avg, am_), (sess.exp_avg_sq, av_)):
            for a in range(0, n, chunk):
                b = min(n, a + chunk)
                d = dev[a:b].cpu().numpy().view(np.uint32)
                if not np.array_equal(d, host[a:b].view(np.uint32)):
                    ok = False
                    break
        verified = ok
        log(f"restored checkpoint == device state after the window: {ok}")

    persist = None
    if args.persist != "none":
        persist = persist_roundtrip(torch, sess, n, args)

    def plain_span(m: int) -> float:
        """Compute-stream ms of m plain steps, started like a window's span
        (from an idle device, right after a host synchronisation)."""
        nonlocal gstep
        torch.cuda.synchronize()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(sess.compute)
        for _ in range(m):
            gstep += 1
            train_step(0, gstep)
        e1.record(sess.compute)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1)

    # checkpoint stall: whole windows with the step after them, no host
    # synchronisation inside, each against a span of the same K + 1 steps
    # without a window taken just before it (both start from an idle device,
    # so the first launch's latency cancels); per window step, median over
    # the pairs
    stall_samples = []
    plain_spans = []
    window_only = []
    if plain_ms:
        window_only = [c / take - plain_ms for take, _, _, c, _, _ in recorded]
        for _ in range(args.stall_windows):
            ref = plain_span(K + 1)
            _, _, _, span = run_window(None, [], post=1)
            plain_spans.append(ref)
            stall_samples.append((span - ref) / K)
        log(f"checkpoint stall per window step over {len(stall_samples)} windows (K steps + the step after, "
            f"each against K + 1 plain steps): {[round(x, 3) for x in stall_samples]} ms")

    pre_ms = upd_ms = cp_ms = comp_ms = gap_ms = 0.0
    alg_fused = alg_pre = alg_d2h = 0
    timed_s = []            # window step of every timed fused launch
    window_alg_bytes = {}   # window step -> algorithmic bytes of its launch (first timed window)
    for take, times, _, c_ms, skips, tail_ms in recorded:
        comp_ms += c_ms
        pre_ms += float(times[:, 0].sum()) + tail_ms
        upd_ms += float(times[:, 1].sum())
        cp_ms += float(times[:, 2].sum())
        gap_ms += float(times[:, 4].sum())
        for s in range(1, take + 1):
            b_s = fused_bytes_measured(n, times[s - 1, 3], bool(skips[s - 1]))
            alg_fused += b_s
            window_alg_bytes.setdefault(s, b_s)
            timed_s.append(s)
            alg_pre += 0 if no_prepass else 2 * n
            # with the HOST_WAIT plan a skipped step's gradients are not sent
            alg_d2h += d2h_bytes(bounds, s) - (2 * int(bounds[s - 1]) if (skips[s - 1] and plan_mode == 1) else 0)
    value = (alg_fused + alg_pre) / ((pre_ms + upd_ms) * 1e-3) / 1e9
    fused_gbs = alg_fused / (upd_ms * 1e-3) / 1e9
    d2h_gbs = alg_d2h / (cp_ms * 1e-3) / 1e9 if cp_ms > 0 else None
    steps_timed = args.steps
    log(f"step+pack {value:.0f} GB/s ({value / HBM_PEAK_GBS:.1%} of 8 TB/s); fused kernel {fused_gbs:.0f} GB/s; "
        f"prepass {pre_ms / steps_timed:.3f} ms/step, update {upd_ms / steps_timed:.3f} ms/step; "
        f"D2H {d2h_gbs or 0:.1f} GB/s")

    timer = SpanTimer(torch, sess, train_step, args.threads, pageable, R)
    model = None
    # staged windows: the worker threads' aggregate rate, taken as workers x
    # the rate of one worker while it copies (an upper bound when they are
    # not all busy at once)
    host_gbs = None
    if pageable:
        hb = sum(st.bytes_host_copied for _, _, st, _, _, _ in recorded)
        hm = sum(st.host_copy_ms for _, _, st, _, _, _ in recorded)
        host_gbs = hb / (hm * 1e-3) / 1e9 * args.copy_threads if hm > 0 else None
    if plain_ms and link_gbs:
        pack_avg = alg_fused / steps_timed - 28 * n
        # the link rate the window's own copies reached (the 1 GiB probe's
        # rate is a little above what a window of 64 MiB copies sustains)
        model = model_params(n, tfb_ms, plain_ms, upd_ms / steps_timed, pack_avg, fused_gbs, d2h_gbs or link_gbs)
        model.update(ring_plan=plan_mode, staging_bytes=staging if pageable else 0, host_gbs=host_gbs or 0.0,
                     link_probe_gbs=link_gbs)
    schemes = None
    if args.schemes and tfb_ms > 0 and (not pageable or args.schemes_pageable):
        schemes = compare_schemes(timer, bounds, K, n, plain_ms, link_gbs, tfb_ms, model, ring_bytes,
                                  sess.cfg.copy_bytes, args)
    plan = None
    if args.plan and model is not None and R == 0:
        plan = compare_plan(timer, bounds, K, n, model, ring_bytes, sess.cfg.copy_bytes,
                            ends if wl["partition"] == "tensors" else None, args)

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(wl, bounds, n, args.seed, args.cpu_seconds, host_cores(), args.grad_dtype)
        log(f"cpu baseline (oracle): {cpu['value']} GB/s on 1 core, {cpu['parallel']['value']} GB/s on "
            f"{cpu['parallel']['cores']} cores, {cpu['sample'].split(' of ')[0]}; {cpu['cpu_model']}")

    per_launch_bytes = alg_fused / steps_timed
    per_launch_ms = upd_ms / steps_timed
    out = {
        "metric": METRIC,
        "value": round(value, 1),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": args.workload, "n_elems": n, "shard": shard, "K": K,
                   "bounds": [int(x) for x in bounds],
                   "ring_bytes": ring_bytes, "copy_bytes": sess.cfg.copy_bytes, "tfb_ms": round(tfb_ms, 3),
                   "fb": fb.describe() if fb is not None else "spin (one wavefront per compute unit)",
                   "host_arena": "pageable via pinned staging" if pageable else "pinned",
                   "host_arena_bytes": int(arena_total), "staging_bytes": staging, "replay_every": R,
                   "placement": args.placement, "ring_plan": args.late_plan, "defer_copies": args.defer_copies,
                   "grad_dtype": args.grad_dtype, "gen_ms": round(gen_ms, 3), "backward_standin_ms": round(bwd_ms, 3),
                   "max_ahead": args.max_ahead, "sync_loss": args.sync_loss,
                   "overflow_test": "none" if args.no_overflow_check else (
                       "caller's found-inf flag" if args.found_inf else (
                           f"{len(scan_edges) - 1} bucket scans beside the backward" if scan_edges is not None
                           else "prepass")),
                   "grad_norm": not no_norm,
                   "state": "fp32 master/m/v, bf16 weights and gradients", "seed": args.seed},
        "hbm_frac": round(value / HBM_PEAK_GBS, 4),
        # the same time with the prepass's second read of the gradients left
        # out of the bytes: the update+pack's bytes over prepass + update
        "hbm_frac_excl_prepass_bytes": round(alg_fused / ((pre_ms + upd_ms) * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
        "elements_per_s": round(n * steps_timed / ((pre_ms + upd_ms) * 1e-3), 1),
        "prepass_ms_per_step": round(pre_ms / steps_timed, 4),
        "update_ms_per_step": round(upd_ms / steps_timed, 4),
        "pre_update_gap_ms_per_step": round(gap_ms / steps_timed, 4),
        # host time inside gockpt_backward_begin + gockpt_step of the timed
        # steps: where the library would make the calling thread wait
        "host_ms_in_library_per_step": {"window": round(host_window_ms, 3),
                                        "plain": round(host_plain_ms, 3) if host_plain_ms is not None else None},
        "d2h_gbs": round(d2h_gbs, 2) if d2h_gbs else None,
        "d2h_link_gbs": round(link_gbs, 2) if link_gbs else None,
        "d2h_frac_of_link": round(d2h_gbs / link_gbs, 4) if (d2h_gbs and link_gbs) else None,
        "device_copy_gbs": round(copy_gbs, 1) if copy_gbs else None,
        "d2h_engine_probe": engine,
        "hbm_probe": probe,
        "fused_frac_of_twin": round(fused_gbs / probe["update_twin_gbs"], 4) if probe else None,
        "compute_ms_per_step": round(comp_ms / steps_timed, 3),
        "plain_ms_per_step": round(plain_ms, 3) if plain_ms else None,
        # the whole checkpoint: K window steps and the step after them minus
        # a span of K + 1 plain steps, per window step (median over the pairs)
        "stall_ms_per_step": round(statistics.median(stall_samples), 3) if stall_samples else None,
        "stall_frac": round(statistics.median(stall_samples) / plain_ms, 4) if stall_samples else None,
        "stall_windows_ms_per_step": [round(x, 3) for x in stall_samples],
        "stall_plain_spans_ms": [round(x, 3) for x in plain_spans],
        "stall_ms_per_checkpoint": round(statistics.median(stall_samples) * K, 2) if stall_samples else None,
        # the timed window steps alone (the step after them not counted)
        "stall_window_only_ms_per_step": round(statistics.median(window_only), 3) if window_only else None,
        "mall_flush": flush_buf is not None,
        "restore_ms": round(restore_ms, 1) if restore_ms is not None else None,
        "restore_element_updates": restore_updates,
        "restore_updates_per_s": round(restore_updates / (restore_ms * 1e-3), 1) if (restore_ms and not R) else None,
        "restore_threads": args.threads,
        "restore_equals_device_state": verified,
        "roofline": {"bound": "hbm", "kernel": "fused_kernel (update + pack)",
                     "achieved": round(per_launch_bytes / (per_launch_ms * 1e-3) / 1e9, 1),
                     "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(per_launch_bytes / (per_launch_ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
                     "bytes_per_launch": int(per_launch_bytes), "ms_per_launch": round(per_launch_ms, 4),
                     "traffic": measured_traffic(args.workload, timed_s) if shard is None else None},
        "cpu_baseline": cpu,
        "persist": persist,
        "schemes": schemes,
        "planner": plan,
        # staged windows: gate kernels the timed windows queued on the copy stream
        "gates_per_window": [int(st.n_gates) for _, _, st, _, _, _ in recorded],
        # bytes the timed windows copied to the host (gradients and state, records not counted)
        "window_d2h_bytes": [int(st.bytes_d2h) for _, _, st, _, _, _ in recorded],
        # staged windows: the worker threads' copies from pinned staging into
        # the pageable arena (GB/s of one worker while copying; workers run in
        # parallel) and the in-window replay's busy time
        "host_copy": ({"bytes": [int(st.bytes_host_copied) for _, _, st, _, _, _ in recorded],
                       "gbs_per_worker": [round(st.bytes_host_copied / (st.host_copy_ms * 1e-3) / 1e9, 2)
                                          if st.host_copy_ms > 0 else None for _, _, st, _, _, _ in recorded],
                       "workers": args.copy_threads,
                       "gbs_aggregate_estimate": round(host_gbs, 2) if host_gbs else None,
                       "replay_ms": [round(st.replay_ms, 1) for _, _, st, _, _, _ in recorded]}
                      if pageable else None),
        "window_ring_bytes": [int(st.bytes_ring) for _, _, st, _, _, _ in recorded],
        "fused_dispatch_steps": dispatch_steps,
        "window_alg_bytes": {str(k): int(v) for k, v in window_alg_bytes.items()},
    }
    sess.close()
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
