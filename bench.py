#!/usr/bin/env python
"""GMC step throughput on one MI355X.

One step is one full iteration of Algorithm 1 for K simulated workers,
gmc_iteration: the worker pass (global momentum + error feedback +
compression + residual for all K workers) and the server pass (sum in
worker order and the apply, w_{t+1} = w_t + update written over w_{t-1}'s
buffer, the two parameter buffers swapping roles every step); GMC+
(lambda > 0) takes gmc_step_detach and gmc_finish.  Inputs are resident in HBM
before the timed region; each step takes the next of a few pre-generated
gradient batches.

Prints one JSON line (stdout): G worker-elements/s (K*d per step), ms/step,
the fraction of HBM peak the step's algorithmic bytes reach, a `roofline`
object for the dominant kernel (the fused worker pass, timed with HIP events
on its own stream inside the timed region) and a `cpu_baseline` object (the
CPU oracle timed on a bounded sample of the same workload).

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload resnet50]
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "GMC step throughput: G worker-elements/s and % of HBM peak, d=25.6M K=16"
UNIT = "G worker-elements/s"
HBM_PEAK_GBS = 8000.0          # MI355X HBM3E peak, GB/s
PMC_SUMMARY = os.path.join(ROOT, "profiles", "topk_fused_vec_resnet50_pmc.txt")
KERNEL_SOURCES = [os.path.join(ROOT, "paper_1905_12948_amd", "csrc", f)
                  for f in ("gmc_kernels.hip", "gmc_internal.h")]

DESCRIPTIONS = {
    "resnet50": "ResNet-50-sized GMC step: d=25,557,032 fp32 in 161 tensors, K=16 workers, global "
                "top-k 0.1% (k=25,558 per worker), Student-t(3) gradients with per-tensor "
                "log-uniform scales in [1e-5,1e-1], beta=0.9, eta=0.1",
    "resnet18": "ResNet-18-sized GMC step: d=11,173,962 fp32 in 62 tensors, K=8, global top-k 1%, "
                "non-IID Gaussian gradients",
    "rbgs": "GMC+ RBGS step: d=25,557,032 fp32, K=8, 1% of 4096-element blocks per step, detached "
            "points w_{t+1,k} = w_{t+1} - lambda eta e_{t+1,k} with lambda=0.5",
    "gpt2": "Transformer-sized GMC step: d=124,439,808 fp32 in 148 tensors, K=8, per-tensor top-k "
            "0.1%, Student-t(4) gradients",
    "tiny": "Tiny GMC step: d=2^20, K=4, global top-k 1%",
    "resnet50_approx": "ResNet-50-sized GMC step with the sampled-threshold top-s of the experiments: "
                       "d=25,557,032, K=16, |S|=d/100 stratified sample, threshold at rank |S|/1024, "
                       "every component at or above it kept",
}


def log(msg: str):
    print("[bench] " + msg, file=sys.stderr, flush=True)


class TimingEvents:
    """HIP events on torch's current stream that only time: created with
    hipEventDisableSystemFence, so that recording one adds no system-scope
    cache write-back and invalidate to the work it brackets (a
    torch.cuda.Event record does, a few microseconds per record)."""

    DISABLE_SYSTEM_FENCE = 0x20000000

    def __init__(self, n: int):
        import ctypes
        self._ct = ctypes
        # the HIP runtime torch has loaded (the soname matches the loaded copy)
        self._hip = ctypes.CDLL("libamdhip64.so.7")
        self._ev = [ctypes.c_void_p() for _ in range(n)]
        for e in self._ev:
            self._ok(self._hip.hipEventCreateWithFlags(ctypes.byref(e), ctypes.c_uint(self.DISABLE_SYSTEM_FENCE)),
                     "hipEventCreateWithFlags")

    @staticmethod
    def _ok(rc: int, what: str):
        if rc != 0:
            raise RuntimeError("%s failed with HIP error %d" % (what, rc))

    def record(self, i: int):
        import torch
        self._ok(self._hip.hipEventRecord(self._ev[i], self._ct.c_void_p(torch.cuda.current_stream().cuda_stream)),
                 "hipEventRecord")

    def elapsed_ms(self, i: int, j: int) -> float:
        self._ok(self._hip.hipEventSynchronize(self._ev[j]), "hipEventSynchronize")
        ms = self._ct.c_float()
        self._ok(self._hip.hipEventElapsedTime(self._ct.byref(ms), self._ev[i], self._ev[j]), "hipEventElapsedTime")
        return ms.value

    def close(self):
        for e in self._ev:
            self._hip.hipEventDestroy(e)
        self._ev = []


def kernel_source_hash():
    """sha256 over the kernel sources, or None where they are not present."""
    h = hashlib.sha256()
    try:
        for p in KERNEL_SOURCES:
            with open(p, "rb") as f:
                h.update(f.read())
    except OSError:
        return None
    return h.hexdigest()


def algorithmic_bytes(wl, msg_len: int, detach: bool, sparse_w: bool = False) -> dict:
    """Bytes one step must move (per step, whole job), and those of the fused
    worker pass alone.  top-s: read g, read e, write e (12 B per worker-
    element); read w_t, w_prev for the momentum term and read w_t, write
    w_{t+1} in the apply (8 B per element each); write (idx, val) and read
    them back in the aggregation (16 B per message entry).  RBGS sends values
    only (8 B).  GMC+'s detached points add one write per worker-element.

    With the sparse momentum term the parameters move only where they change:
    w_t - w_prev is +0 off the components the last server pass changed, so
    the worker pass reads that pass's bitmap (d/8 B) and w_t, w_prev at most
    at the K message entries (8 B each); the server pass reads the old
    bitmap, writes the new one and reads w_t, writes w_{t+1} at most at the
    old and the new entries (2 x 8 B each).  GMC+'s detached points still
    read w_t whole (4 B per element)."""
    K, d = wl.K, wl.d
    rbgs = wl.compressor == "rbgs"
    per_msg = 8 if rbgs else 16
    sent = K * msg_len
    if sparse_w:
        w_worker = d // 8 + 8 * sent + (4 * d if detach else 0)
        w_server = 2 * (d // 8) + 16 * sent
    else:
        w_worker, w_server = 8 * d, 8 * d
    points = 4 * K * d if detach else 0
    step = 12 * K * d + w_worker + w_server + per_msg * sent + points
    fused = 12 * K * d + w_worker + (4 * sent if rbgs else 0) + points
    return {"step": step, "fused": fused}


def survey_bytes(wl, msg_len: int, detach: bool) -> int:
    """The step's algorithmic bytes with dense parameter traffic: read g,
    read e, write e (12 B per worker-element); read w_t and w_{t-1} for the
    momentum term, read w_t and write w_{t+1} in the apply (16 B per
    element); write each message entry and read it back in the aggregation
    (16 B for an (index, value) pair, 8 B for an RBGS value).  GMC+ adds its
    detached points, one write per worker-element."""
    K, d = wl.K, wl.d
    per_msg = 8 if wl.compressor == "rbgs" else 16
    return 12 * K * d + 16 * d + per_msg * K * msg_len + (4 * K * d if detach else 0)


def host_cpu() -> dict:
    """The host the CPU baseline ran on: logical CPUs and the model name."""
    model = None
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        usable = len(os.sched_getaffinity(0))
    except (AttributeError, OSError):
        usable = None
    return {"nproc": os.cpu_count(), "usable_cpus": usable, "model": model}


def read_pmc_summary(sparse_w: bool = True):
    """Per-dispatch HBM traffic of the fused kernel from the committed
    rocprofv3 counter summary, scaled by the copy-kernel calibration; None if
    absent, taken on different kernel sources or in the other momentum mode."""
    if not os.path.exists(PMC_SUMMARY):
        return None
    kv = {}
    with open(PMC_SUMMARY) as f:
        for line in f:
            if "=" in line and not line.lstrip().startswith("#"):
                k, v = line.split("=", 1)
                kv[k.strip()] = v.strip()
    try:
        src = kernel_source_hash()
        if src is None or kv.get("kernel_source_sha256") != src:
            return None
        if kv.get("sparse_momentum", "0") != ("1" if sparse_w else "0"):
            return None
        fs = float(kv["copy_bytes"]) / (float(kv["copy_fetch_kib"]) * 1024.0)
        ws = float(kv["copy_bytes"]) / (float(kv["copy_write_kib"]) * 1024.0)
        return (float(kv["fused_fetch_kib"]) * 1024.0 * fs + float(kv["fused_write_kib"]) * 1024.0 * ws)
    except (KeyError, ValueError, ZeroDivisionError):
        return None


def cpu_baseline(wl, workers: int, steps: int, lam: float = 0.0) -> dict:
    """The CPU oracle (single-threaded C, as it stands) on a bounded sample
    of the workload: `workers` of the K workers at the full d for `steps`
    iterations, with host-generated inputs of the same recipe (and GMC+'s
    detached points when lam > 0)."""
    import numpy as np
    import oracle
    import synth
    import dataclasses
    sub = dataclasses.replace(wl, K=workers)
    seg = sub.topk_segments() if sub.compressor == "topk_seg" else None
    orc = oracle.GmcOracle(sub.d, workers, sub.compressor if sub.compressor in ("rbgs", "approx") else "topk",
                           sub.ratio, sub.beta, sub.eta, seed=sub.seed, seg_off=seg, block=sub.block, lam=lam)
    w = sub.w0()
    wp = w.copy()
    err = np.zeros((workers, sub.d), np.float32)
    batches = [sub.grads(t) for t in range(steps)]
    t0 = time.perf_counter()
    for t in range(steps):
        idx, val, ln = orc.step(w, wp, batches[t], err)
        delta = orc.aggregate(idx, val, ln)
        wn = w.copy()
        orc.apply(wn, delta)
        if lam > 0.0:
            orc.detach(wn, err)
        wp, w = w, wn
    dt = time.perf_counter() - t0
    host = host_cpu()
    return {"value": workers * sub.d * steps / dt / 1e9, "unit": UNIT, "cores": 1, "kind": "oracle",
            "sample": "%d of the %d workers at the full d=%d for %d steps (oracle compression, "
                      "aggregation of those %d messages and apply each step), %.1f s of CPU time"
                      % (workers, wl.K, wl.d, steps, workers, dt),
            "threads_used": 1, "host_nproc": host["nproc"], "host_usable_cpus": host["usable_cpus"],
            "host_cpu": host["model"],
            "note": "1 core used: the oracle is single-threaded C (-O2, no fp contraction)"}


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=30)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="resnet50", choices=sorted(DESCRIPTIONS))
    ap.add_argument("--grad-batches", type=int, default=4)
    ap.add_argument("--margin", type=int, default=None,
                    help="rank of the speculative threshold in quarters of k (default 4)")
    ap.add_argument("--lam", type=float, default=None,
                    help="GMC+ detach coefficient (default 0.5 for the rbgs workload, else 0: plain GMC)")
    ap.add_argument("--dense-momentum", action="store_true",
                    help="read w_t and w_prev everywhere (no GMC_OPT_SPARSE_MOMENTUM)")
    ap.add_argument("--cpu-workers", type=int, default=2)
    ap.add_argument("--cpu-steps", type=int, default=2)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--change-list", type=int, default=None, choices=(0, 1, 2),
                    help="GMC_OPT_CHANGE_LIST: 0 by size (default), 1 always, 2 never")
    ap.add_argument("--in-place", action="store_true",
                    help="one parameter buffer updated in place (gmc_iteration_inplace; GMC_OPT_CHANGE_LIST 3): "
                         "top-s only")
    ap.add_argument("--force-full", action="store_true",
                    help="every top-s selection of the timed steps on the full-data path (GMC_OPT_FORCE_FULL_SELECT), "
                         "to profile the fallback path")
    ap.add_argument("--calib", action="store_true",
                    help="also run the plain copy kernel (memory-counter calibration)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: the K workers are simulated on a single MI355X and "
              "nothing in this build uses a second GPU (run with --gpus 1)", file=sys.stderr)
        sys.exit(2)

    import torch
    import synth
    import synth.device as sdev
    from paper_1905_12948_amd import Gmc
    from paper_1905_12948_amd.gmc import calib_copy, calib_stream

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(2)
    dev = torch.device("cuda:0")
    wl = synth.workload(args.workload)
    d, K = wl.d, wl.K
    seg = wl.topk_segments().tolist() if wl.compressor == "topk_seg" else None
    lam = args.lam if args.lam is not None else (0.5 if wl.compressor == "rbgs" else 0.0)
    detach = lam > 0.0
    gm = Gmc(d, K, wl.compressor, wl.ratio, wl.beta, wl.eta, seed=wl.seed, segments=seg,
             block=wl.block if wl.compressor == "rbgs" else None, lam=lam)
    if args.margin is not None:
        from paper_1905_12948_amd import GMC_OPT_CAND_MARGIN
        gm.set_option(GMC_OPT_CAND_MARGIN, args.margin)
    if args.force_full:
        from paper_1905_12948_amd import GMC_OPT_FORCE_FULL_SELECT
        gm.set_option(GMC_OPT_FORCE_FULL_SELECT, 1)
    if args.in_place and (wl.compressor == "rbgs" or args.dense_momentum or lam):
        print("--in-place is for top-s with the sparse momentum term and no detached points", file=sys.stderr)
        sys.exit(2)
    if args.change_list is not None or args.in_place:
        from paper_1905_12948_amd import GMC_OPT_CHANGE_LIST
        gm.set_option(GMC_OPT_CHANGE_LIST, 3 if args.in_place else args.change_list)
    # the bench keeps w untouched between the server pass and the next worker
    # pass and swaps the two buffers, as the sparse momentum term requires
    sparse_w = not args.dense_momentum
    if sparse_w:
        from paper_1905_12948_amd import GMC_OPT_SPARSE_MOMENTUM
        gm.set_option(GMC_OPT_SPARSE_MOMENTUM, 1)
    log("workload %s: d=%d K=%d %s ratio=%g; generating %d gradient batches on the GPU"
        % (wl.name, d, K, wl.compressor, wl.ratio, args.grad_batches))
    w = sdev.w0(wl, dev)
    wp = w.clone()
    # K per-worker rows packed with a 128-byte-aligned pitch (sdev.rows)
    err = sdev.rows(K, d, dev, zero=True)
    G = [sdev.grads(wl, t, dev) for t in range(args.grad_batches)]
    idx, val, ln = gm.alloc_messages(dev)
    wk = sdev.rows(K, d, dev) if detach else None   # GMC+ detached points w_{t+1,k}
    if args.calib:
        cal_src = torch.ones(1 << 28, dtype=torch.float32, device=dev)     # 1 GiB
        cal_dst = torch.empty_like(cal_src)
    torch.cuda.synchronize()

    # w_t and w_{t-1} live in two buffers whose roles swap every step:
    # gmc_aggregate_apply writes w_{t+1} = w_t + update over w_{t-1}'s buffer
    bufs = [w, wp]
    step_no = [0]

    def one_step():
        cur, prev = bufs[step_no[0] % 2], bufs[(step_no[0] + 1) % 2]
        if args.in_place:  # one buffer: w_{t+1} over w_t, w_{t-1} kept as the change list
            gm.iteration_inplace(w, w if step_no[0] == 0 else None, G[step_no[0] % len(G)], err, idx, val, ln)
        elif detach:
            gm.step(cur, prev, G[step_no[0] % len(G)], err, idx, val, ln, w_k=wk)
            gm.finish(idx, val, ln, cur, prev, err=err, w_k=wk)
        else:  # worker and server pass in one call: w_{t+1} over w_{t-1}'s buffer
            gm.iteration(cur, prev, G[step_no[0] % len(G)], err, idx, val, ln)
        step_no[0] += 1

    log("warmup %d steps" % args.warmup)
    for _ in range(args.warmup):
        one_step()
    torch.cuda.synchronize()
    stats0 = gm.stats()
    gm.profile(["fused_vec"])

    log("timing %d steps" % args.steps)
    # the value comes from the host clock around the whole timed region; the
    # only events in it are the library's pair around each worker pass (the
    # roofline's kernel time): every event record is a barrier packet in the
    # queue, 1-3 us of the step
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        one_step()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    prof = gm.profile_read()
    stats1 = gm.stats()
    gm.profile([])
    # iteration 0 on its own: a fresh context of the same configuration
    # (every kernel is loaded by now, and the context allocates its scratch
    # when it is created, before the timed call) takes one step from e = 0
    # and w_t = w_{t-1}, with no previous threshold: the seed kernel's
    # threshold from a strided sample of u stands in for it, and only a
    # selection whose candidates miss the count takes the full-data path
    g0 = Gmc(d, K, wl.compressor, wl.ratio, wl.beta, wl.eta, seed=wl.seed, segments=seg,
             block=wl.block if wl.compressor == "rbgs" else None, lam=lam)
    if sparse_w:
        g0.set_option(GMC_OPT_SPARSE_MOMENTUM, 1)
    err.zero_()
    bufs[1].copy_(bufs[0])
    torch.cuda.synchronize()
    fev = TimingEvents(2)
    fev.record(0)
    if detach:
        g0.step(bufs[0], bufs[1], G[0], err, idx, val, ln, w_k=wk)
        g0.finish(idx, val, ln, bufs[0], bufs[1], err=err, w_k=wk)
    else:
        g0.iteration(bufs[0], bufs[1], G[0], err, idx, val, ln)
    fev.record(1)
    torch.cuda.synchronize()
    first = {"ms": round(fev.elapsed_ms(0, 1), 4), "full_data_selections": g0.stats()["full_data"]}
    g0.close()
    # the full-data selection path (the fallback when the candidates cannot
    # prove they hold the top k): one step from the same state with every
    # selection forced onto it
    full = None
    if wl.compressor in ("topk", "topk_seg"):
        from paper_1905_12948_amd import GMC_OPT_FORCE_FULL_SELECT
        g1 = Gmc(d, K, wl.compressor, wl.ratio, wl.beta, wl.eta, seed=wl.seed, segments=seg, lam=lam)
        g1.set_option(GMC_OPT_FORCE_FULL_SELECT, 1)
        err.zero_()
        bufs[1].copy_(bufs[0])
        torch.cuda.synchronize()
        fev.record(0)
        g1.step(bufs[0], bufs[1], G[0], err, idx, val, ln, w_k=wk if detach else None)
        fev.record(1)
        torch.cuda.synchronize()
        full = {"ms": round(fev.elapsed_ms(0, 1), 4), "full_data_selections": g1.stats()["full_data"],
                "what": "gmc_step alone, every selection on the full-data path"}
        g1.close()
    if args.calib:
        for _ in range(3):
            calib_copy(cal_dst, cal_src)
        torch.cuda.synchronize()
    # the stream ceiling of the worker pass's access pattern: the plain stream
    # e += g over the same K rows (top-s without detached points only; the
    # residuals are no longer needed)
    stream = None
    if wl.compressor != "rbgs" and not detach:
        for _ in range(2):
            calib_stream(err, G[0])
        reps = 5
        fev.record(0)
        for _ in range(reps):
            calib_stream(err, G[0])
        fev.record(1)
        torch.cuda.synchronize()
        stream_ms = fev.elapsed_ms(0, 1) / reps
        stream = {"kernel": "calib_stream_kernel", "bytes": 12 * K * d, "avg_ms": round(stream_ms, 4),
                  "achieved": round(12 * K * d / (stream_ms * 1e-3) / 1e9, 1)}

    fev.close()
    ms_step = elapsed * 1e3 / args.steps
    msg_len = int(round(float(ln.double().mean().item())))  # varies per worker for the sampled threshold
    # relative communication cost of the last timed step (Section 5.2):
    # values the K workers send plus K times the components of the server's
    # update, over the 2 K d values dense exchanges would move (top-s also
    # sends an index with each value)
    ln_h = [int(x) for x in ln.cpu().tolist()]
    if wl.compressor == "rbgs":
        support = ln_h[0]  # every worker sends the same blocks
    else:
        support = int(torch.unique(torch.cat([idx[k, :ln_h[k]] for k in range(K)])).numel())
    rcc = (sum(ln_h) + K * support) / (2.0 * K * d)
    ab = algorithmic_bytes(wl, msg_len, detach, sparse_w)
    fused_ms_total, fused_n = prof["fused_vec"]
    fused_ms = fused_ms_total / max(fused_n, 1)
    achieved = ab["fused"] / (fused_ms * 1e-3) / 1e9
    traffic = read_pmc_summary(sparse_w) if (wl.name == "resnet50" and not detach) else None
    roofline = {"kernel": "topk_fused_vec_kernel" if wl.compressor != "rbgs" else "rbgs_vec_kernel",
                "bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(achieved / HBM_PEAK_GBS, 4),
                "traffic": None if traffic is None else int(traffic),
                "alg_bytes_per_launch": ab["fused"], "avg_ms": round(fused_ms, 4)}
    if stream is not None:
        # the worker pass's time against the plain stream of its pattern
        stream["kernel_time_frac"] = round(stream_ms / fused_ms, 4)
        roofline["stream_ceiling"] = stream
    value = K * d / (ms_step * 1e-3) / 1e9
    sel = {k: stats1[k] - stats0[k] for k in ("from_candidates", "full_data", "candidates", "count_errors",
                                              "sparse_momentum_steps", "sparse_applies")}
    dense_bytes = survey_bytes(wl, msg_len, detach)
    out = {
        "metric": METRIC if wl.name == "resnet50" else METRIC.split(",")[0] + ", " + wl.name,
        "value": round(value, 2), "unit": UNIT, "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_step, 4),
        "first_step": first,
        "full_data_step": full,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": DESCRIPTIONS[wl.name], "d": d, "K": K, "compressor": wl.compressor,
                   "ratio": wl.ratio, "lambda": lam, "message_len": msg_len, "grad_batches": len(G),
                   "sparse_momentum": sparse_w, "forced_full_data": bool(args.force_full),
                   "in_place": bool(args.in_place),
                   "rcc": round(rcc, 7), "update_support": support},
        # the step's algorithmic bytes with dense parameter traffic (12 B per
        # worker-element, 16 B per element, 16 B per message entry) over
        # 8 TB/s; the sparse accounting (parameters moved only where they
        # change) is beside it
        "hbm_peak_frac": round(dense_bytes / (ms_step * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
        "alg_bytes_per_step": dense_bytes,
        "sparse_accounting": {"alg_bytes_per_step": ab["step"],
                              "hbm_peak_frac": round(ab["step"] / (ms_step * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)},
        "selection": sel,
        "roofline": roofline,
    }
    if not args.no_cpu_baseline:
        log("cpu baseline: oracle on %d workers x %d steps" % (args.cpu_workers, args.cpu_steps))
        del G
        torch.cuda.empty_cache()
        out["cpu_baseline"] = cpu_baseline(wl, args.cpu_workers, args.cpu_steps, lam)
    gm.close()
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
