#!/usr/bin/env python3
"""Benchmark: batched Chamfer distance forward + backward on one MI355X.

A step is one pass of the whole path over one batch of synthetic clouds that
are already resident in HBM: nearest neighbours both ways (cd_forward), the
Chamfer reduction and the F-score at every threshold of the workload (one
cd_metrics call) and the backward to both clouds (cd_backward).  The default
workload is B=16, N=M=16384 points sampled on random 200-triangle meshes with
F-score at tau = 0.005, 0.01, 0.02.

Throughput is credited 2*B*N*M directed pair-evaluations per step (one per
query/target pair in each direction).  The roofline object prices the
dominant call (cd_forward: the fused nearest-neighbour search kernel and its
merge kernel, timed with HIP events around every cd_forward call on the launch
stream) at 9 FP32 operations per directed
pair-evaluation against the MI355X FP32 vector peak of 157.3 TFLOP/s.

Prints ONE JSON line.  Single GPU only.
"""
from __future__ import annotations

import argparse
import ctypes
import json
import os
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "Chamfer fwd+bwd pair-evals/sec and ms/call at B=16, N=M=16384; % FP32 VALU peak"
PEAK_FP32_TFLOPS = 157.3          # MI355X FP32 vector, 256 CU x 2.4 GHz x 256 flop/clk
FLOPS_PER_PAIR = 9                # 3 sub + 3 mul + 2 add + 1 min per directed pair-eval
EXECUTED_FLOPS_PER_PAIR = 10      # per computed distance: 3 sub, 3 mul, 2 add, row + column min
# Sources of cd_forward's kernels and the flags they are built with.
FORWARD_SOURCES = ("paper_1911_05063_amd/csrc/nn_search.hip", "paper_1911_05063_amd/build.py")


def parse_args():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=100,
                    help="untimed steps after the settle phase")
    ap.add_argument("--settle-ms", type=float, default=200.0,
                    help="before the warm-up, run steps until this much GPU time has passed "
                         "(the GPU clock ramps up over the first ~50 ms of work; reported as "
                         "settle_ms / settle_steps)")
    ap.add_argument("--no-per-config", action="store_true",
                    help="skip the per-workload figures of the five Chamfer workloads")
    ap.add_argument("--workload", type=int, default=3, help="workload number 1..5 (default 3)")
    ap.add_argument("--path", choices=("chamfer", "mesh", "p2s", "emd"), default="chamfer",
                    help="chamfer: the Chamfer step on the workload (default); mesh: the mesh "
                         "reconstruction loss step (surface sampling -> Chamfer -> vertex "
                         "gradients) on 16 meshes of 200 triangles, 16384 samples each; "
                         "p2s: the point-to-surface loss step on 16 deformed icospheres of "
                         "5120 faces against 16384 points each; emd: the approximate EMD step "
                         "(50 Sinkhorn iterations + backward) on the sphere workload")
    ap.add_argument("--no-cpu-baseline", action="store_true", help="skip the CPU oracle timing")
    ap.add_argument("--cpu-items", type=int, default=0,
                    help="batch items in the CPU-oracle sample (0 = all items)")
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="repeat the CPU-oracle sample until this much time has passed")
    ap.add_argument("--ingest-pmc", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"),
                    help="read two rocprofv3 --pmc runs (FETCH_SIZE, WRITE_SIZE; each with "
                         "--calib-copy 256), write profiles/traffic_mesh_b16_n16384.json, exit")
    ap.add_argument("--ingest-valu", nargs="+", metavar="K=DIR",
                    help="read rocprofv3 --pmc runs of SQ_INSTS_VALU, SQ_ACTIVE_INST_VALU and "
                         "SQ_THREAD_CYCLES_VALU, one per workload k (bench.py --workload k), "
                         "write profiles/counters_cd_forward_valu.json, exit")
    ap.add_argument("--calib-copy", type=int, default=0, metavar="MIB",
                    help="after the timed steps, fill then copy an MIB-MiB device buffer once: "
                         "reference kernels of known size for HBM-counter calibration")
    return ap.parse_args()


def _sources_sha256(kernel_sources):
    import hashlib
    h = hashlib.sha256()
    for src in kernel_sources:
        with open(os.path.join(ROOT, src), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def library_sources_sha256():
    """sha256 over the library's sources (csrc/, the build script, the C
    header): names the build a measurement or a profile describes."""
    import glob
    srcs = sorted(glob.glob(os.path.join(ROOT, "paper_1911_05063_amd", "csrc", "*")))
    srcs += [os.path.join(ROOT, "paper_1911_05063_amd", "build.py"),
             os.path.join(ROOT, "include", "cd.h")]
    return _sources_sha256([os.path.relpath(p, ROOT) for p in srcs])


def ingest_pmc(fetch_dir, write_dir, calib_mib=256):
    """Per-dispatch FETCH_SIZE / WRITE_SIZE (KiB) of cd_forward's kernels, each
    scaled by what the counter reads for the calibration copy of calib_mib MiB."""
    import csv
    import glob
    from collections import defaultdict

    def averages(d):
        paths = glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True)
        if not paths:
            raise SystemExit(f"no counter_collection.csv under {d}")
        acc = defaultdict(list)
        with open(paths[0]) as f:
            for row in csv.DictReader(f):
                acc[row["Kernel_Name"]].append(float(row["Counter_Value"]))
        return {k: sum(v) / len(v) for k, v in acc.items()}

    def pick(avg, key):
        hits = [v for k, v in avg.items() if key in k]
        if len(hits) != 1:
            raise SystemExit(f"expected one kernel matching {key!r}, found {len(hits)}")
        return hits[0]

    fa, wa = averages(fetch_dir), averages(write_dir)
    ref_kib = calib_mib * 1024.0
    fs = ref_kib / pick(fa, "copyBuffer")
    ws = ref_kib / pick(wa, "copyBuffer")
    raw = {k: {"FETCH_SIZE": pick(fa, k), "WRITE_SIZE": pick(wa, k)} for k in FORWARD_KERNELS}
    fetch = sum(r["FETCH_SIZE"] for r in raw.values()) * fs * 1024.0
    write = sum(r["WRITE_SIZE"] for r in raw.values()) * ws * 1024.0
    rec = {"kernel_source_sha256": _sources_sha256(FORWARD_SOURCES),
           "workload": "mesh_b16_n16384 (B=16, N=M=16384)",
           "launch": "cd_forward = key_fill_kernel + search_kernel + merge_kernel",
           "hbm_bytes_per_launch": round(fetch + write),
           "fetch_bytes_per_launch": round(fetch), "write_bytes_per_launch": round(write),
           "per_kernel_kib_raw": {k: {c: round(v, 1) for c, v in r.items()} for k, r in raw.items()},
           "calibration": {"reference": f"__amd_rocclr_copyBuffer of {calib_mib} MiB",
                           "fetch_scale": round(fs, 4), "write_scale": round(ws, 4)},
           "algorithmic_bytes_per_launch": 20 * 16 * (16384 + 16384)}
    out = os.path.join(ROOT, "profiles", "traffic_mesh_b16_n16384.json")
    with open(out, "w") as f:
        json.dump(rec, f, indent=1)
    print(json.dumps(rec))


def traffic_record(kernel_sources):
    """HBM bytes per cd_forward from the committed counter summary, or None when
    the kernel sources changed since the counters were taken."""
    path = os.path.join(ROOT, "profiles", "traffic_mesh_b16_n16384.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f)
    if rec.get("kernel_source_sha256") != _sources_sha256(kernel_sources):
        return None
    return rec


VALU_RECORD = os.path.join(ROOT, "profiles", "counters_cd_forward_valu.json")
FORWARD_KERNELS = ("key_fill_kernel", "search_kernel", "merge_kernel")
CLOCK_GHZ, N_CU, FMA_LANES_PER_CU = 2.4, 256, 128


def _pmc_averages(d):
    """Per-kernel mean of each counter over the dispatches of one rocprofv3 --pmc run."""
    import csv
    import glob
    from collections import defaultdict
    paths = glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True)
    if not paths:
        raise SystemExit(f"no counter_collection.csv under {d}")
    acc = defaultdict(lambda: defaultdict(list))
    with open(paths[0]) as f:
        for row in csv.DictReader(f):
            acc[row["Counter_Name"]][row["Kernel_Name"]].append(float(row["Counter_Value"]))
    return {c: {k: sum(v) / len(v) for k, v in per.items()} for c, per in acc.items()}


def ingest_valu(specs):
    """VALU lane-operations per cd_forward call, per workload, from one
    rocprofv3 --pmc run each (K=DIR: bench.py --workload K under rocprofv3)."""
    import synth
    rec = {"kernel_source_sha256": _sources_sha256(FORWARD_SOURCES),
           "sources": list(FORWARD_SOURCES),
           "counters": "SQ_INSTS_VALU, SQ_ACTIVE_INST_VALU, SQ_THREAD_CYCLES_VALU (chip totals, "
                       "mean per dispatch)",
           "lane_ops": "SQ_THREAD_CYCLES_VALU summed over the forward's kernels: VALU "
                       "instructions times their active lanes",
           "workloads": {}}
    for spec in specs:
        k, d = spec.split("=", 1)
        w = synth.WORKLOADS[int(k)]
        avg = _pmc_averages(d)
        per = {}
        for kern in FORWARD_KERNELS:
            hit = {c: [v for name, v in avg[c].items() if kern in name]
                   for c in ("SQ_INSTS_VALU", "SQ_ACTIVE_INST_VALU", "SQ_THREAD_CYCLES_VALU")}
            if any(len(v) != 1 for v in hit.values()):
                raise SystemExit(f"workload {k}: expected one kernel matching {kern!r}")
            per[kern] = {c: v[0] for c, v in hit.items()}
        lane_ops = sum(p["SQ_THREAD_CYCLES_VALU"] for p in per.values())
        srch = per["search_kernel"]
        rec["workloads"][w.name] = {
            "per_kernel": per, "lane_ops_per_call": lane_ops,
            "search_lane_utilisation": srch["SQ_THREAD_CYCLES_VALU"] / (64.0 * srch["SQ_ACTIVE_INST_VALU"]),
            "search_valu_insts_per_computed_pair": srch["SQ_INSTS_VALU"] * 64.0 / (w.B * w.N * w.M)}
    with open(VALU_RECORD, "w") as f:
        json.dump(rec, f, indent=1)
    print(json.dumps(rec))


def valu_record():
    """The committed VALU counter record, or None when cd_forward's sources
    changed since it was taken."""
    if not os.path.exists(VALU_RECORD):
        return None
    with open(VALU_RECORD) as f:
        rec = json.load(f)
    if rec.get("kernel_source_sha256") != _sources_sha256(FORWARD_SOURCES):
        return None
    return rec


def forward_fractions(B, N, M, fwd_ms, rec, name):
    """The three roofline fractions of one cd_forward call of fwd_ms:
    credited (9 flop per directed pair-evaluation, 2 B N M of them), executed
    (10 flop per computed distance, B N M of them: 3 sub, 1 mul, 2 FMA, the
    row and the column minimum) and the VALU issue fraction from the counter
    record (lane-operations over 128 lanes per CU-clock at 2.4 GHz)."""
    t = fwd_ms * 1e-3
    peak = PEAK_FP32_TFLOPS * 1e12
    credited = FLOPS_PER_PAIR * 2.0 * B * N * M / t / peak
    executed = EXECUTED_FLOPS_PER_PAIR * float(B) * N * M / t / peak
    issue = None
    if rec is not None and name in rec["workloads"]:
        lane_ops = rec["workloads"][name]["lane_ops_per_call"]
        issue = lane_ops / (t * CLOCK_GHZ * 1e9 * N_CU * FMA_LANES_PER_CU)
    return credited, executed, issue


def _loaded_hip_runtime():
    """Path of the HIP runtime this process has loaded (torch's), so that the
    events below live in the same runtime as the streams they are recorded on."""
    with open("/proc/self/maps") as f:
        for line in f:
            path = line.split()[-1]
            if os.path.basename(path).startswith("libamdhip64.so"):
                return path
    raise RuntimeError("the HIP runtime is not loaded (import torch and use the GPU first)")


class HipEvent:
    """A HIP timing event recorded without the system-scope release fence
    (hipEventDisableSystemFence).  Recording a default event (what
    torch.cuda.Event creates) writes back and invalidates the L2 cache: about
    2.4 us of GPU time between two calls, against about 1.2 us for this one;
    the intervals measured are the same.  Same methods as torch.cuda.Event."""
    _hip = None
    DISABLE_SYSTEM_FENCE = 0x20000000

    @classmethod
    def _runtime(cls):
        if cls._hip is None:
            hip = ctypes.CDLL(_loaded_hip_runtime())
            hip.hipEventCreateWithFlags.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_uint]
            hip.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
            hip.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p,
                                                ctypes.c_void_p]
            hip.hipEventDestroy.argtypes = [ctypes.c_void_p]
            cls._hip = hip
        return cls._hip

    def __init__(self):
        self._h = ctypes.c_void_p()
        rc = self._runtime().hipEventCreateWithFlags(ctypes.byref(self._h), self.DISABLE_SYSTEM_FENCE)
        if rc != 0:
            raise RuntimeError(f"hipEventCreateWithFlags failed ({rc})")

    def record(self, stream):
        rc = self._hip.hipEventRecord(self._h, ctypes.c_void_p(stream.cuda_stream))
        if rc != 0:
            raise RuntimeError(f"hipEventRecord failed ({rc})")

    def elapsed_time(self, end):
        ms = ctypes.c_float()
        rc = self._hip.hipEventElapsedTime(ctypes.byref(ms), self._h, end._h)
        if rc != 0:
            raise RuntimeError(f"hipEventElapsedTime failed ({rc})")
        return ms.value

    def __del__(self):
        try:
            if self._h and HipEvent._hip is not None:
                HipEvent._hip.hipEventDestroy(self._h)
                self._h = ctypes.c_void_p()
        except Exception:  # interpreter shutdown: nothing left to release
            pass


class Timing:
    """Result of timed_steps: per-step events, total ms of the timed steps,
    their wall seconds, and the settle phase (GPU ms, steps)."""

    def __init__(self, events, total_ms, wall_s, settle_ms, settle_steps):
        self.events, self.total_ms, self.wall_s = events, total_ms, wall_s
        self.settle_ms, self.settle_steps = settle_ms, settle_steps


def settle(one, stream, min_ms, max_wall_s=5.0):
    """Clock settle: run steps (no events) in rounds of 5 until at least
    min_ms of GPU time has passed between the first launch and the last
    completion, or max_wall_s of wall time.  Returns (GPU ms, steps)."""
    import torch
    if min_ms <= 0:
        return 0.0, 0
    a, b = HipEvent(), HipEvent()
    n, t0 = 0, time.perf_counter()
    a.record(stream)
    while True:
        for _ in range(5):
            one(None)
        n += 5
        b.record(stream)
        torch.cuda.synchronize()
        ms = a.elapsed_time(b)
        if ms >= min_ms or time.perf_counter() - t0 >= max_wall_s:
            return ms, n


def timed_steps(one, n_marks, steps, warmup, stream, settle_ms):
    """Settle, warm-up, then exactly `steps` timed steps between two
    synchronizations.

    one(ev) runs a step and records the n_marks events of `ev` (None: no
    events).  Each recorded event costs about a microsecond of GPU time, so
    the timed steps record only the events their figures need.  The GPU
    clock ramps up over the first ~50 ms of work, so the steps first run
    until settle_ms of GPU time has passed (settle()), then `warmup` more.
    Every event is created before that, so the timed steps follow the
    warm-up's synchronization without an idle gap: after a few milliseconds
    idle the clock drops and needs tens of calls to ramp back up."""
    import torch

    evs = [[HipEvent() for _ in range(n_marks)] for _ in range(steps)]
    start, stop = HipEvent(), HipEvent()
    s_ms, s_n = settle(one, stream, settle_ms)
    for _ in range(warmup):
        one(None)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    start.record(stream)
    for k in range(steps):
        one(evs[k] if n_marks else None)
    stop.record(stream)
    torch.cuda.synchronize()
    return Timing(evs, start.elapsed_time(stop), time.perf_counter() - t0, s_ms, s_n)


class Step:
    """Preallocated buffers and the C-ABI calls of one step (marshalling only)."""

    def __init__(self, X, Y, taus):
        import torch
        import paper_1911_05063_amd as cd
        self.torch = torch
        self.lib = cd.library()
        self.cd = cd
        self.X, self.Y = X, Y
        B, N, M = X.shape[0], X.shape[1], Y.shape[1]
        self.B, self.N, self.M = B, N, M
        dev = X.device
        f32, i32 = torch.float32, torch.int32
        self.dxy = torch.empty((B, N), dtype=f32, device=dev)
        self.ixy = torch.empty((B, N), dtype=i32, device=dev)
        self.dyx = torch.empty((B, M), dtype=f32, device=dev)
        self.iyx = torch.empty((B, M), dtype=i32, device=dev)
        self.ws_bytes = int(self.lib.cd_workspace_bytes(B, N, M))
        self.ws = torch.empty(self.ws_bytes, dtype=torch.uint8, device=dev)
        self.bws_bytes = int(self.lib.cd_backward_workspace_bytes(B, N, M))
        self.bws = torch.empty(self.bws_bytes, dtype=torch.uint8, device=dev)
        self.chamfer = torch.empty(B, dtype=f32, device=dev)
        self.taus = list(taus)
        self.fs = [torch.empty((len(self.taus), B), dtype=f32, device=dev) for _ in range(3)]
        self.tau_arr = (ctypes.c_float * len(self.taus))(*self.taus)
        self.tau_ptr = ctypes.cast(self.tau_arr, ctypes.c_void_p)
        self.grad_out = torch.ones(B, dtype=f32, device=dev)
        self.gX = torch.empty_like(X)
        self.gY = torch.empty_like(Y)
        self.stream = torch.cuda.current_stream(dev)
        self.s = ctypes.c_void_p(self.stream.cuda_stream)
        P = lambda t: ctypes.c_void_p(t.data_ptr())  # noqa: E731
        self.p = {k: P(v) for k, v in dict(X=X, Y=Y, dxy=self.dxy, ixy=self.ixy, dyx=self.dyx,
                                           iyx=self.iyx, ws=self.ws, bws=self.bws,
                                           ch=self.chamfer,
                                           go=self.grad_out, gX=self.gX, gY=self.gY,
                                           f=self.fs[0], pr=self.fs[1], rc=self.fs[2]).items()}

    def _ok(self, st, what):
        if st != 0:
            raise RuntimeError(f"{what}: {self.lib.cd_status_string(st).decode()}: "
                               f"{self.lib.cd_last_error().decode()}")

    def forward(self):
        p = self.p
        self._ok(self.lib.cd_forward(self.B, self.N, self.M, p["X"], p["Y"], p["dxy"], p["ixy"],
                                     p["dyx"], p["iyx"], p["ws"], self.ws_bytes, self.s), "cd_forward")

    def reduce_fscore(self):
        """Chamfer and F-score at every tau: one cd_metrics launch."""
        p = self.p
        self._ok(self.lib.cd_metrics(self.B, self.N, self.M, p["dxy"], p["dyx"], 1.0, 1.0,
                                     self.tau_ptr, len(self.taus), p["ch"], p["f"], p["pr"],
                                     p["rc"], self.s), "cd_metrics")

    def backward(self):
        p = self.p
        self._ok(self.lib.cd_backward(self.B, self.N, self.M, p["go"], 1.0, 1.0, p["X"], p["Y"],
                                      p["ixy"], p["iyx"], p["gX"], p["gY"], p["bws"],
                                      self.bws_bytes, self.s), "cd_backward")


def repeat_for(run_once, seconds):
    """Run run_once() until `seconds` have passed (at least once); returns
    (repetitions, elapsed seconds)."""
    reps, t0 = 0, time.perf_counter()
    while True:
        run_once()
        reps += 1
        dt = time.perf_counter() - t0
        if dt >= seconds:
            return reps, dt


def cpu_model():
    """The host CPU's model name (first processor in /proc/cpuinfo)."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def time_cpu_oracle(X, Y, taus, items, seconds):
    """The CPU oracle (as it stands) on `items` batch items of the workload:
    nearest neighbours both ways, Chamfer, F-score at each tau, backward;
    repeated for about `seconds` with all of the oracle's threads, then on
    one item with one thread for about half as long."""
    import numpy as np
    import oracle
    oracle.nn_one_way(X[:1, :8], Y[:1, :8])  # load + spin up the thread pool

    def leg(n_items, secs):
        Xs, Ys = X[:n_items], Y[:n_items]

        def once():
            r = oracle.forward_all(Xs, Ys, taus)
            oracle.backward(np.ones(n_items), Xs, Ys, r["idx_xy"], r["idx_yx"])

        reps, dt = repeat_for(once, secs)
        return 2.0 * n_items * X.shape[1] * Y.shape[1] * reps / dt, reps, dt

    what = (f"float32 nearest neighbours both ways, Chamfer, F-score at {len(taus)} thresholds "
            f"and backward")
    threads = oracle.threads()
    rate, reps, dt = leg(items, seconds)
    oracle.set_threads(1)
    try:
        rate1, reps1, dt1 = leg(1, seconds / 2)
    finally:
        oracle.set_threads(threads)
    try:
        affinity = len(os.sched_getaffinity(0))
    except AttributeError:
        affinity = os.cpu_count()
    return {"value": rate, "unit": "pair-evals/s", "cores": threads,
            "kind": "oracle", "seconds": round(dt, 3), "cpu_model": cpu_model(),
            "host_cpus": os.cpu_count(), "cpus_available": affinity,
            "sample": (f"{items} of {X.shape[0]} batch items (N={X.shape[1]}, M={Y.shape[1]}), "
                       f"{reps} times: {what}, OpenMP over queries ({threads} threads)"),
            "single_thread": {"value": rate1, "unit": "pair-evals/s", "cores": 1,
                              "seconds": round(dt1, 3),
                              "sample": f"1 batch item (N={X.shape[1]}, M={Y.shape[1]}), "
                                        f"{reps1} times: {what}, one thread"}}


def mesh_step_bench(args):
    """The mesh reconstruction loss step (Sec. 2.1 sampling feeding the Sec. 2.5
    Chamfer loss): choose faces, sample points, Chamfer + F-score against a
    target cloud, Chamfer backward, sampling backward to the vertices."""
    import numpy as np
    import torch
    import paper_1911_05063_amd as cd
    import synth

    B, T, S, M = 16, 200, 16384, 16384
    V_np, F_np = synth.triangle_soup(B, T, 3)
    _, Y_np = synth.generate("mesh", B, 1, M, 30)
    u_np, r1_np, r2_np = synth.uniforms(B, S, 31)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    g = lambda a: torch.from_numpy(np.array(a, copy=True)).to(dev)  # noqa: E731
    V, F, Y, u, r1, r2 = (g(a) for a in (V_np, F_np, Y_np, u_np, r1_np, r2_np))
    lib = cd.library()
    P = lambda t: ctypes.c_void_p(t.data_ptr())  # noqa: E731
    stream = torch.cuda.current_stream(dev)
    st = ctypes.c_void_p(stream.cuda_stream)
    mws = torch.empty(int(lib.cd_mesh_workspace_bytes(B, 3 * T, T, S)), dtype=torch.uint8, device=dev)
    fidx = torch.empty((B, S), dtype=torch.int32, device=dev)
    X = torch.empty((B, S, 3), dtype=torch.float32, device=dev)
    step = Step(X, Y, (0.005, 0.01, 0.02))
    gV = torch.empty_like(V)

    def ok(rc, what):
        if rc != 0:
            raise RuntimeError(f"{what}: {lib.cd_last_error().decode()}")

    def one(ev=None):
        if ev is not None:
            ev[0].record(stream)
        ok(lib.cd_mesh_sample_faces(B, 3 * T, T, P(V), P(F), S, P(u), P(fidx), P(mws),
                                    mws.numel(), st), "faces")
        ok(lib.cd_mesh_sample_points(B, 3 * T, T, P(V), P(F), S, P(fidx), P(r1), P(r2), P(X), st),
           "points")
        if ev is not None:
            ev[1].record(stream)
        step.forward()
        step.reduce_fscore()
        step.backward()
        if ev is not None:
            ev[2].record(stream)
        ok(lib.cd_mesh_sample_backward(B, 3 * T, T, P(F), S, P(fidx), P(r1), P(r2), P(step.gX),
                                       P(gV), P(mws), mws.numel(), st), "sample backward")
        if ev is not None:
            ev[3].record(stream)

    tm = timed_steps(one, 0, args.steps, args.warmup, stream, args.settle_ms)
    ms = tm.total_ms / args.steps
    nb = min(args.steps, 50)
    # per-call breakdown, after the timed steps
    evs = timed_steps(one, 4, nb, args.warmup, stream, args.settle_ms / 4).events
    samp = statistics.mean(e[0].elapsed_time(e[1]) for e in evs)
    cham = statistics.mean(e[1].elapsed_time(e[2]) for e in evs)
    sbwd = statistics.mean(e[2].elapsed_time(e[3]) for e in evs)
    pairs = 2.0 * B * S * M
    out = {"metric": "mesh reconstruction loss step pair-evals/sec (sampling + Chamfer fwd+bwd + "
                     "sampling bwd)",
           "value": pairs / (ms * 1e-3), "unit": "pair-evals/s", "n_gpus": 1,
           "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms,
           "settle_ms": tm.settle_ms, "settle_steps": tm.settle_steps,
           "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32",
           "data": "synthetic",
           "library_sha256": library_sources_sha256(),
           "config": {"workload": "mesh_sampling_b16_t200_s16384", "B": B, "triangles": T,
                      "samples": S, "M": M, "taus": [0.005, 0.01, 0.02]},
           "ms_per_call": {"sample_faces+points": samp, "chamfer_fwd_metrics_bwd": cham,
                           "sample_backward": sbwd, "breakdown_steps": nb},
           "pct_fp32_valu_peak": 100.0 * FLOPS_PER_PAIR * pairs / (ms * 1e-3) / (PEAK_FP32_TFLOPS * 1e12)}
    print(json.dumps(out), flush=True)


# Point-to-surface pair function, counted on the straightforward evaluation
# (an FMA counts 2): v = p - a (3); s, t and the normal offset h, three dot
# products (15); u = 1 - s - t (2); inside test (3); three clamped segment
# distances of 18 each (54); v - e0 for the third edge (3); minimum of the
# edges (2); h^2 (1); selection (1); comparison with the best so far (1).
P2S_FLOPS_PER_PAIR = 85


def time_cpu_p2s(P, V, F, items, points, seconds):
    """The oracle's point-to-surface forward + backward on a bounded sample:
    the first `points` points of each of the first `items` items, repeated
    for about `seconds`."""
    import numpy as np
    import oracle
    Ps, Vs, Fs = P[:items, :points], V[:items], F[:items]

    def once():
        dist, fidx, _ = oracle.p2s_forward(Ps, Vs, Fs)
        oracle.p2s_backward(Ps, Vs, Fs, fidx, np.full(fidx.shape, 1.0 / points))

    reps, dt = repeat_for(once, seconds)
    pairs = float(items) * points * F.shape[1] * reps
    return {"value": pairs / dt, "unit": "point-triangle pair-evals/s", "cores": oracle.threads(),
            "kind": "oracle", "seconds": round(dt, 3),
            "sample": f"{items} items x {points} points x {F.shape[1]} faces, {reps} times, "
                      f"forward + backward, OpenMP over points"}


def p2s_step_bench(args):
    """The point-to-surface loss step (Sec. 2.5): cd_p2s_forward, the per-item
    mean (cd_reduce), cd_p2s_backward to the points and the vertices."""
    import numpy as np
    import torch
    import paper_1911_05063_amd as cd
    import synth

    w = synth.P2S_WORKLOAD
    P_np, V_np, F_np = synth.p2s_workload(w.B, w.S, w.level, w.seed)
    B, S, nv, nf = w.B, w.S, V_np.shape[1], F_np.shape[1]
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    g = lambda a: torch.from_numpy(np.array(a, copy=True)).to(dev)  # noqa: E731
    P, V, F = g(P_np), g(V_np), g(F_np)
    lib = cd.library()
    ptr = lambda t: ctypes.c_void_p(t.data_ptr())  # noqa: E731
    stream = torch.cuda.current_stream(dev)
    st = ctypes.c_void_p(stream.cuda_stream)
    ws = torch.empty(int(lib.cd_p2s_workspace_bytes(B, S, nv, nf)), dtype=torch.uint8, device=dev)
    dist = torch.empty((B, S), dtype=torch.float32, device=dev)
    fidx = torch.empty((B, S), dtype=torch.int32, device=dev)
    loss = torch.empty(B, dtype=torch.float32, device=dev)
    gdist = torch.full((B, S), 1.0 / S, dtype=torch.float32, device=dev)
    gP = torch.empty_like(P)
    gV = torch.empty_like(V)

    def ok(rc, what):
        if rc != 0:
            raise RuntimeError(f"{what}: {lib.cd_last_error().decode()}")

    def one(ev=None):
        if ev is not None:
            ev[0].record(stream)
        ok(lib.cd_p2s_forward(B, S, nv, nf, ptr(P), ptr(V), ptr(F), ptr(dist), ptr(fidx), ptr(ws),
                              ws.numel(), st), "forward")
        if ev is not None:
            ev[1].record(stream)
        ok(lib.cd_reduce(B, S, S, ptr(dist), ptr(dist), ctypes.c_float(1.0), ctypes.c_float(0.0),
                         ptr(loss), st), "reduce")
        ok(lib.cd_p2s_backward(B, S, nv, nf, ptr(P), ptr(V), ptr(F), ptr(fidx), ptr(gdist),
                               ptr(gP), ptr(gV), ptr(ws), ws.numel(), st), "backward")

    print(f"[bench] {w.name}: B={B} S={S} nv={nv} nf={nf} steps={args.steps} "
          f"warmup={args.warmup}", file=sys.stderr, flush=True)
    tm = timed_steps(one, 2, args.steps, args.warmup, stream, args.settle_ms)
    ms = tm.total_ms / args.steps
    fwd = statistics.mean(e[0].elapsed_time(e[1]) for e in tm.events)
    rest = ms - fwd
    pairs = float(B) * S * nf
    achieved = P2S_FLOPS_PER_PAIR * pairs / (fwd * 1e-3) / 1e12
    out = {"metric": "point-to-surface loss step point-triangle pair-evals/sec "
                     "(forward + mean + backward to points and vertices)",
           "value": pairs / (ms * 1e-3), "unit": "point-triangle pair-evals/s", "n_gpus": 1,
           "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms,
           "settle_ms": tm.settle_ms, "settle_steps": tm.settle_steps,
           "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32",
           "data": "synthetic",
           "library_sha256": library_sources_sha256(),
           "config": {"workload": w.name, "B": B, "S": S, "nv": nv, "nf": nf},
           "ms_per_call": {"cd_p2s_forward": fwd, "reduce+backward": rest},
           "roofline": {"bound": "alu", "kernel": "cd_p2s_forward (face records + search + merge)",
                        "achieved": achieved, "peak": PEAK_FP32_TFLOPS, "unit": "TFLOP/s",
                        "frac": achieved / PEAK_FP32_TFLOPS, "traffic": None,
                        "work_per_launch": f"{P2S_FLOPS_PER_PAIR} flop x {pairs:.4g} "
                                           f"point-triangle pairs"}}
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = time_cpu_p2s(P_np, V_np, F_np, B, S, args.cpu_seconds)
    print(json.dumps(out), flush=True)


# Sinkhorn half-update pair function (an FMA counts 2): the distance (3 sub,
# 3 mul, 2 add), its square root (1), the exponent (fma: 2), the batch
# maximum (1), the shifted exponent (sub 1, exp2 1) and the sum (1).
EMD_FLOPS_PER_PAIR = 15
EMD_ITERS, EMD_EPS = 50, (0.5, 0.01)


def time_cpu_emd(X, Y, seconds):
    """The oracle's scheduled Sinkhorn + backward, one batch item at a time
    (items 0, 1, ... in turn) for about `seconds`."""
    import numpy as np
    from oracle import emd_oracle
    done = [0]

    def once():
        b = done[0] % X.shape[0]
        cost, F, G = emd_oracle.sinkhorn(X[b:b + 1], Y[b:b + 1], EMD_EPS[0], EMD_EPS[1], EMD_ITERS)
        emd_oracle.backward(X[b:b + 1], Y[b:b + 1], F, G, EMD_EPS[1], np.ones(1))
        done[0] += 1

    items, dt = repeat_for(once, seconds)
    pairs = float(items) * X.shape[1] * Y.shape[1] * (2 * EMD_ITERS + 3)
    return {"value": pairs / dt, "unit": "Sinkhorn pair-evals/s", "cores": 1, "kind": "oracle",
            "seconds": round(dt, 3),
            "sample": f"{items} items x {X.shape[1]} x {Y.shape[1]} points, {EMD_ITERS} iterations "
                      f"+ cost + backward (NumPy float64, dense cost matrix)"}


def emd_step_bench(args):
    """The approximate-EMD loss step (Sec. 2.5): cd_emd_forward (scheduled
    Sinkhorn iterations and the transport cost) and cd_emd_backward."""
    import numpy as np
    import torch
    import paper_1911_05063_amd as cd
    import synth

    w = synth.WORKLOADS[2]
    X_np, Y_np = synth.workload(2)
    B, N, M = w.B, w.N, w.M
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    X = torch.from_numpy(X_np).to(dev)
    Y = torch.from_numpy(Y_np).to(dev)
    lib = cd.library()
    ptr = lambda t: ctypes.c_void_p(t.data_ptr())  # noqa: E731
    stream = torch.cuda.current_stream(dev)
    st = ctypes.c_void_p(stream.cuda_stream)
    ws = torch.empty(int(lib.cd_emd_workspace_bytes(B, N, M)), dtype=torch.uint8, device=dev)
    f = torch.empty((B, N), dtype=torch.float32, device=dev)
    g = torch.empty((B, M), dtype=torch.float32, device=dev)
    cost = torch.empty(B, dtype=torch.float32, device=dev)
    go = torch.ones(B, dtype=torch.float32, device=dev)
    gX, gY = torch.empty_like(X), torch.empty_like(Y)

    def ok(rc, what):
        if rc != 0:
            raise RuntimeError(f"{what}: {lib.cd_last_error().decode()}")

    def one(ev=None):
        if ev is not None:
            ev[0].record(stream)
        ok(lib.cd_emd_forward(B, N, M, ptr(X), ptr(Y), EMD_EPS[0], EMD_EPS[1], EMD_ITERS, 0,
                              ptr(f), ptr(g), ptr(cost), ptr(ws), ws.numel(), st), "forward")
        if ev is not None:
            ev[1].record(stream)
        ok(lib.cd_emd_backward(B, N, M, ptr(X), ptr(Y), ptr(f), ptr(g), EMD_EPS[1], ptr(go),
                               ptr(gX), ptr(gY), ptr(ws), ws.numel(), st), "backward")

    print(f"[bench] emd on {w.describe()} iters={EMD_ITERS} eps={EMD_EPS} steps={args.steps} "
          f"warmup={args.warmup}", file=sys.stderr, flush=True)
    tm = timed_steps(one, 2, args.steps, args.warmup, stream, args.settle_ms)
    ms = tm.total_ms / args.steps
    fwd = statistics.mean(e[0].elapsed_time(e[1]) for e in tm.events)
    bwd = ms - fwd
    pairs = float(B) * N * M * (2 * EMD_ITERS + 3)
    lse_pairs = float(B) * N * M * 2 * EMD_ITERS
    # The forward is dominated by the 2 * iters log-sum-exp passes; price them
    # (the cost pass is a further B N M pairs inside the same interval).
    achieved = EMD_FLOPS_PER_PAIR * lse_pairs / (fwd * 1e-3) / 1e12
    out = {"metric": "approximate-EMD step Sinkhorn pair-evals/sec (50 iterations + cost + backward)",
           "value": pairs / (ms * 1e-3), "unit": "Sinkhorn pair-evals/s", "n_gpus": 1,
           "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms,
           "settle_ms": tm.settle_ms, "settle_steps": tm.settle_steps,
           "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32",
           "data": "synthetic",
           "library_sha256": library_sources_sha256(),
           "config": {"workload": w.name, "B": B, "N": N, "M": M, "iters": EMD_ITERS,
                      "eps": list(EMD_EPS)},
           "ms_per_call": {"cd_emd_forward": fwd, "cd_emd_backward": bwd},
           "roofline": {"bound": "alu", "kernel": "cd_emd_forward (lse passes + cost pass)",
                        "achieved": achieved, "peak": PEAK_FP32_TFLOPS, "unit": "TFLOP/s",
                        "frac": achieved / PEAK_FP32_TFLOPS, "traffic": None,
                        "work_per_launch": f"{EMD_FLOPS_PER_PAIR} flop x {lse_pairs:.4g} "
                                           f"log-sum-exp pair terms"}}
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = time_cpu_emd(X_np, Y_np, args.cpu_seconds)
    print(json.dumps(out), flush=True)


def main():
    args = parse_args()
    if args.ingest_pmc:
        ingest_pmc(*args.ingest_pmc)
        return
    if args.ingest_valu:
        ingest_valu(args.ingest_valu)
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported "
              f"(the batch items are independent: shard them across GPUs).", file=sys.stderr)
        sys.exit(2)
    if args.path == "emd":
        emd_step_bench(args)
        return
    if args.path == "p2s":
        p2s_step_bench(args)
        return
    if args.path == "mesh":
        mesh_step_bench(args)
        return
    chamfer_bench(args)


def chamfer_step_on(k):
    """Workload k's clouds on cuda:0 and a Step over them (inputs resident in HBM)."""
    import torch
    import synth
    X_np, Y_np = synth.workload(k)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    step = Step(torch.from_numpy(X_np).to(dev), torch.from_numpy(Y_np).to(dev),
                synth.WORKLOADS[k].taus)
    return step, X_np, Y_np


def measure_chamfer(step, steps, warmup, settle_ms, breakdown_steps):
    """The Chamfer step (cd_forward, cd_metrics, cd_backward) timed: `steps`
    steps with events around every cd_forward (the roofline's launch
    duration), then a pass of breakdown_steps with four events per step for
    the metrics and backward calls (its own settle: the clock drops while
    its events are created)."""

    def one_step(ev=None):
        if ev is not None:
            ev[0].record(step.stream)
        step.forward()
        if ev is not None:
            ev[1].record(step.stream)
        step.reduce_fscore()
        if ev is not None and len(ev) > 2:
            ev[2].record(step.stream)
        step.backward()
        if ev is not None and len(ev) > 2:
            ev[3].record(step.stream)

    tm = timed_steps(one_step, 2, steps, warmup, step.stream, settle_ms)
    bd = timed_steps(one_step, 4, breakdown_steps, warmup, step.stream, settle_ms / 4)
    return {"timing": tm, "ms_per_step": tm.total_ms / steps,
            "fwd": [e[0].elapsed_time(e[1]) for e in tm.events],
            "red": [e[1].elapsed_time(e[2]) for e in bd.events],
            "bwd": [e[2].elapsed_time(e[3]) for e in bd.events]}


def max_in_degree(step):
    """The backward's scatter contention after a step: over all items, the
    largest number of senders whose nearest neighbour is one receiver (Y
    points onto an x, X points onto a y), from the step's index outputs
    (copied to the host after the timed region)."""
    import numpy as np
    step.torch.cuda.synchronize()
    ixy, iyx = step.ixy.cpu().numpy(), step.iyx.cpu().numpy()
    onto_x = max(int(np.bincount(r, minlength=step.N).max()) for r in iyx)
    onto_y = max(int(np.bincount(r, minlength=step.M).max()) for r in ixy)
    return {"onto_x": onto_x, "onto_y": onto_y}


def config_figures(w, m, rec, step):
    """Per-workload figures of one measure_chamfer() result."""
    fwd = statistics.mean(m["fwd"])
    credited, executed, issue = forward_fractions(w.B, w.N, w.M, fwd, rec, w.name)
    return {"B": w.B, "N": w.N, "M": w.M, "steps": len(m["timing"].events),
            "max_in_degree": max_in_degree(step),
            "ms_per_step": m["ms_per_step"],
            "pair_evals_per_s": 2.0 * w.B * w.N * w.M / (m["ms_per_step"] * 1e-3),
            "ms_per_call": {"forward": fwd, "metrics": statistics.mean(m["red"]),
                            "backward": statistics.mean(m["bwd"])},
            "frac": credited, "executed_frac": executed, "valu_issue_frac": issue}


def per_config(args, main_k, main_fig, rec):
    """Every Chamfer workload's figures (GPU only), about 50 ms of timed
    steps each; the benchmark's own workload reuses its main figures."""
    import torch
    import synth
    out = {}
    for k in sorted(synth.WORKLOADS):
        w = synth.WORKLOADS[k]
        if k == main_k:
            out[w.name] = main_fig
            continue
        step, _, _ = chamfer_step_on(k)
        probe_ms, probe_n = settle(lambda ev=None: (step.forward(), step.reduce_fscore(),
                                                    step.backward()),
                                   step.stream, 100.0)
        n = int(min(200, max(10, 50.0 / (probe_ms / probe_n))))
        print(f"[bench] per-config {w.name}: {n} steps", file=sys.stderr, flush=True)
        m = measure_chamfer(step, n, 5, 20.0, min(n, 50))
        out[w.name] = config_figures(w, m, rec, step)
        del step
        torch.cuda.empty_cache()
    return out


def chamfer_bench(args):
    import torch
    import synth

    w = synth.WORKLOADS[args.workload]
    step, X_np, Y_np = chamfer_step_on(args.workload)
    dev = step.X.device
    print(f"[bench] {w.describe()} steps={args.steps} warmup={args.warmup} "
          f"settle_ms={args.settle_ms}", file=sys.stderr, flush=True)
    m = measure_chamfer(step, args.steps, args.warmup, args.settle_ms, min(args.steps, 50))
    tm, fwd, red, bwd = m["timing"], m["fwd"], m["red"], m["bwd"]

    if args.calib_copy > 0:
        n = args.calib_copy * (1 << 20) // 4
        src = torch.empty(n, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        src.fill_(1.0)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    B, N, M = w.B, w.N, w.M
    pairs = 2.0 * B * N * M
    ms_per_step = m["ms_per_step"]
    value = pairs / (ms_per_step * 1e-3)
    fwd_avg_s = statistics.mean(fwd) * 1e-3
    achieved = FLOPS_PER_PAIR * pairs / fwd_avg_s / 1e12
    rec = valu_record()
    main_fig = config_figures(w, m, rec, step)
    out = {
        "metric": METRIC,
        "value": value,
        "unit": "pair-evals/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "settle_ms": tm.settle_ms,
        "settle_steps": tm.settle_steps,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": w.name, "kind": w.kind, "B": B, "N": N, "M": M,
                   "taus": list(w.taus), "seed": w.seed},
        "library_sha256": library_sources_sha256(),
        "ms_per_call": {"forward": statistics.mean(fwd), "forward_median": statistics.median(fwd),
                        "reduce_fscore": statistics.mean(red), "backward": statistics.mean(bwd),
                        "fwd_bwd": ms_per_step, "breakdown_steps": len(red)},
        "pct_fp32_valu_peak": 100.0 * FLOPS_PER_PAIR * value / (PEAK_FP32_TFLOPS * 1e12),
        "wall_s": tm.wall_s,
        "roofline": {"bound": "alu",
                     "kernel": "cd_forward (key_fill_kernel + search_kernel + merge_kernel)",
                     "achieved": achieved, "peak": PEAK_FP32_TFLOPS, "unit": "TFLOP/s",
                     "frac": achieved / PEAK_FP32_TFLOPS, "traffic": None,
                     "executed_frac": main_fig["executed_frac"],
                     "valu_issue_frac": main_fig["valu_issue_frac"],
                     "frac_note": "frac credits 9 flop per directed pair-evaluation (2 B N M); "
                                  "executed_frac counts the 10 flop per distance the fused "
                                  "kernel computes (B N M); valu_issue_frac is VALU "
                                  "lane-operations (counter record) over 128 lanes per "
                                  "CU-clock at 2.4 GHz",
                     "algorithmic_bytes": 12.0 * B * (N + M) + 8.0 * B * (N + M),
                     "work_per_launch": f"{FLOPS_PER_PAIR} flop x {pairs:.4g} directed pair-evals"},
    }
    tr = traffic_record(FORWARD_SOURCES) if args.workload == 3 else None
    if tr is not None:
        out["roofline"]["traffic"] = tr["hbm_bytes_per_launch"]
    if not args.no_per_config:
        del step
        torch.cuda.empty_cache()
        out["per_config"] = per_config(args, args.workload, main_fig, rec)
    if not args.no_cpu_baseline:
        items = args.cpu_items if args.cpu_items > 0 else B
        print(f"[bench] CPU oracle baseline on {items} item(s)", file=sys.stderr, flush=True)
        out["cpu_baseline"] = time_cpu_oracle(X_np, Y_np, w.taus, min(items, B),
                                              args.cpu_seconds)
    else:
        out["cpu_baseline"] = None
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
