"""Throughput of the GaLore 2 gradient-subspace hot path on one MI355X.

One step is one pass of the whole path over a batch of same-shape gradients:
the randomized-SVD subspace update (sketch, power iterations with
re-orthonormalisation, small SVD, projector), the projection R = P^T A, the
low-rank Adam step and the back-projected weight update.

Workload (default): the 64 gate/up projection gradients of a Llama-7B-shaped
model, 4096 x 11008 each, stored bf16 and computed in fp32, power-law planted
spectrum s_i = (i+1)^-0.7 plus 1e-4 Gaussian noise; rank r = 1024,
oversampling p = 32, q = 2 power iterations; Adam beta = (0.9, 0.999),
eps = 1e-8, lr = 1e-3, scale alpha = 0.25. Inputs are synthetic, generated on
the device and resident in HBM before the timed region starts.

Prints ONE JSON line. `value` is subspace updates per second (each matrix of
the batch gets one update, one projection, one Adam step and one weight update
per step). Per-stage times come from HIP events recorded on the stream the
library launches on; the Adam stage is one kernel launch, so its duration gives
the achieved HBM bandwidth of that kernel.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0         # MI355X HBM3E, GB/s
FP32_MFMA_PEAK_TFS = 157.3    # MI355X dense fp32 matrix, TFLOP/s
FP64_MFMA_PEAK_TFS = 78.6     # MI355X dense fp64 matrix, TFLOP/s
BF16_MFMA_PEAK_TFS = 2500.0   # MI355X dense bf16 matrix, TFLOP/s
INT8_MFMA_PEAK_TOPS = 5000.0  # MI355X dense int8 matrix, TOP/s
ADAM_BYTES_PER_ELEM = 24      # read R, M, V; write M, V, N (fp32)

# kernel classes of the roofline: launch classes (traced stages or outer calls)
# that run one kernel each, the kernel's symbol and its source file (a stored
# counter reading is used only while that source is unchanged)
KERNEL_CLASSES = {
    "products": (("product_A", "product_At"), "gemm_bf16x3_kernel", "bf16x3.hip"),
    "gram": (("gram",), "gram_i8_kernel", "gram_i8.hip"),
    "triangular": (("triangular",), None, "gemm.hip"),
    "projector": (("projector",), None, "gemm.hip"),
    "project": (("project",), None, "gemm.hip"),
    "project_back": (("project_back",), None, "gemm.hip"),
    "adam": (("adam",), "adam_flat_kernel", "elementwise.hip"),
}
CSRC = os.path.join(ROOT, "paper_2504_20437_amd", "csrc")


def kernel_class(cls, dtype):
    members, sym, src = KERNEL_CLASSES[cls]
    if cls == "products" and dtype == "f32":      # fp32-stored G: the fp32 GEMM kernel
        sym, src = None, "gemm.hip"
    return members, sym, src


def source_hash(fname):
    import hashlib
    h = hashlib.sha256()
    for f in (fname, "common.hpp"):
        with open(os.path.join(CSRC, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def workload_key(cls, args):
    # matrices per launch: the batch, or one chunk of it with --streams
    return "%s:%dx%dx%d:r%d:p%d:q%d:%s" % (cls, args.batch // max(1, args.streams), args.m, args.n, args.r, args.p,
                                          args.q, args.dtype)


def write_traffic(args):
    """Per-launch HBM bytes of each kernel class from two rocprofv3 counter
    runs. FETCH_SIZE and WRITE_SIZE (KiB per dispatch) are scaled by what they
    read for the plain device-to-device copy of --copy-probe-mib MiB that the
    profiled run made first (a copy reads and writes exactly that many bytes)."""
    import csv

    def load(path, counter):
        rows = [r for r in csv.DictReader(open(path)) if r["Counter_Name"] == counter]
        copies = [float(r["Counter_Value"]) for r in rows if "copyBuffer" in r["Kernel_Name"]]
        if not copies or args.copy_probe_mib <= 0:
            raise SystemExit("%s: no copy-probe dispatch (run the profiled bench with --copy-probe-mib)" % path)
        factor = args.copy_probe_mib * 1024.0 / max(copies)      # true KiB per counted KiB
        return rows, factor

    frows, ff = load(args.write_traffic[0], "FETCH_SIZE")
    wrows, fw = load(args.write_traffic[1], "WRITE_SIZE")
    try:
        with open(args.traffic_json) as f:
            out = json.load(f)
    except (OSError, ValueError):
        out = {}
    for cls in KERNEL_CLASSES:
        _, sym, src = kernel_class(cls, args.dtype)
        if sym is None:
            continue
        fv = [float(r["Counter_Value"]) for r in frows if sym in r["Kernel_Name"]]
        wv = [float(r["Counter_Value"]) for r in wrows if sym in r["Kernel_Name"]]
        if not fv or not wv:
            continue
        fetch = sum(fv) / len(fv) * ff * 1024.0
        write = sum(wv) / len(wv) * fw * 1024.0
        out[workload_key(cls, args)] = {
            "kernel": sym, "dispatches": len(fv), "fetch_bytes": round(fetch), "write_bytes": round(write),
            "bytes_per_launch": round(fetch + write), "fetch_factor": round(ff, 4), "write_factor": round(fw, 4),
            "source_sha256": source_hash(src), "command": args.command,
        }
    with open(args.traffic_json, "w") as f:
        json.dump(out, f, indent=1, sort_keys=True)
        f.write("\n")
    print(json.dumps({k: v["bytes_per_launch"] for k, v in out.items()}))


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=3)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--m", type=int, default=4096)
    ap.add_argument("--n", type=int, default=11008)
    ap.add_argument("--batch", type=int, default=64)
    ap.add_argument("--r", type=int, default=1024)
    ap.add_argument("--p", type=int, default=32)
    ap.add_argument("--q", type=int, default=2)
    ap.add_argument("--dtype", default="bf16", choices=["bf16", "f32"])
    ap.add_argument("--streams", type=int, default=1,
                    help="split the batch into this many equal chunks, each on its own stream (default "
                         "priority), so that one chunk's latency-bound stages overlap another's products")
    ap.add_argument("--cpu-baseline", type=int, default=1,
                    help="time the oracle on the host (0: no, 1: one matrix of the workload, 2: also q = 1, the "
                         "other two shapes of the model and one thread on a 2048x5461 matrix; minutes of host time)")
    ap.add_argument("--whole-model", type=int, default=1,
                    help="also time a subspace update and a projected Adam step of all 224 Llama-7B-shaped "
                         "matrices (0/1; needs the default 4096x11008 batch of 64 on one stream)")
    ap.add_argument("--configs", type=int, default=1,
                    help="also time the smaller workloads of the same family (single 256x688 matrix, the 60M-, "
                         "350M- and 1B-shaped layer sets) as extra keys (0/1)")
    ap.add_argument("--extras", type=int, default=1,
                    help="also time the schedule, the low-bit projector, the exact SVD and the 8-bit Adam (0/1; 0 "
                         "for short profiling runs)")
    ap.add_argument("--roofline-kernel", default="auto", choices=["auto"] + sorted(KERNEL_CLASSES))
    ap.add_argument("--copy-probe-mib", type=int, default=0,
                    help="before the workload, copy a buffer of this many MiB device to device once (a "
                         "plain copy of known size, to calibrate rocprofv3 FETCH_SIZE / WRITE_SIZE)")
    ap.add_argument("--traffic-json", default=os.path.join(ROOT, "profiles", "traffic.json"),
                    help="per-launch HBM bytes from rocprofv3 counters (optional)")
    ap.add_argument("--write-traffic", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                    help="no benchmark: read the counter_collection.csv of a rocprofv3 --pmc FETCH_SIZE run "
                         "and of a --pmc WRITE_SIZE run of this script (same workload flags, with "
                         "--copy-probe-mib), and record the per-launch HBM bytes of each kernel class in "
                         "--traffic-json")
    ap.add_argument("--command", default="", help="with --write-traffic: the profiling command, recorded")
    return ap.parse_args()


def _cpu_model() -> str:
    """The host CPU as /proc/cpuinfo names it, with family/model/stepping, cache
    and the number of CPUs this process may run on."""
    fields = {}
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if ":" not in line:
                    continue
                key, val = (x.strip() for x in line.split(":", 1))
                if key in ("model name", "cpu family", "model", "stepping", "cache size") and key not in fields:
                    fields[key] = val
    except OSError:
        pass
    try:
        usable = len(os.sched_getaffinity(0))
    except (AttributeError, OSError):
        usable = os.cpu_count()
    return "%s (family %s, model %s, stepping %s, cache %s; %s CPUs usable by this process)" % (
        fields.get("model name", "?"), fields.get("cpu family", "?"), fields.get("model", "?"),
        fields.get("stepping", "?"), fields.get("cache size", "?"), usable)


def _oracle_path(oracle, gi, m, n, r, p, q, dtype, seed):
    """One matrix through the oracle's whole path; seconds per stage (each
    printed to stderr as it ends)."""
    import numpy as np

    s = min(m, n)
    G = gi.store(gi.planted_gradient(m, n, gi.spectrum_power(s, 0.7), 1e-4, seed=seed), dtype)
    W = gi.weights(m, n, seed=seed + 1).astype(np.float64)
    f32 = lambda x: float(np.float32(x))
    t = [time.perf_counter()]

    def mark(stage):
        t.append(time.perf_counter())
        print("bench: oracle %dx%d r=%d q=%d %s: %.2f s" % (m, n, r, q, stage, t[-1] - t[-2]), file=sys.stderr,
              flush=True)
    P, _, _ = oracle.rsvd_update(G.exact, r, p, q, gi.sketch_seed(0))
    mark("update")
    R = oracle.project(P, G.exact)
    mark("projection")
    Mz = np.zeros_like(R)
    _, _, N = oracle.adam(R, Mz, Mz, f32(0.9), f32(0.999), f32(1e-8), 1)
    mark("Adam")
    oracle.project_back(P, N, W, f32(1e-3), f32(0.25))
    mark("back-projection")
    d = [b - a for a, b in zip(t, t[1:])]
    return {"update_s": round(d[0], 3), "project_s": round(d[1], 3), "adam_s": round(d[2], 4),
            "project_back_s": round(d[3], 3), "total_s": round(sum(d), 3)}


def cpu_baseline(args):
    """The oracle timed on the host on a bounded sample of the workload: one of
    its matrices (same shape, spectrum and storage, r, p, q), run through the
    whole path: subspace update, projection, Adam step and weight update, each
    stage timed. With --cpu-baseline 2 also: the same matrix on one thread,
    q = 1, the 4096x4096 and 11008x4096 shapes of the same model, and a
    2048x5461 matrix on all threads and on one (a few minutes of host time;
    not part of the default run)."""
    import oracle

    import galore_inputs as gi

    m, n, r, p, q = args.m, args.n, args.r, args.p, args.q
    threads = oracle.num_threads()
    main = _oracle_path(oracle, gi, m, n, r, p, q, args.dtype, 7000)
    dt = main["total_s"]
    out = {
        "value": 1.0 / dt,
        "unit": "updates/s",
        "cores": threads,
        "kind": "oracle",
        "sample": "one %dx%d %s matrix of the workload, r=%d p=%d q=%d, whole path (update, projection, "
                  "Adam step, weight update) once: %.1f s" % (m, n, args.dtype, r, p, q, dt),
        "stage_s": main,
        "cpu_model": _cpu_model(),
    }
    if (m, n) == (4096, 11008):
        # every term of the oracle's update and step scales with l = max(m, n) at
        # fixed s and k, so a 4096x4096 matrix costs about 4096/11008 of this one
        # and an 11008x4096 matrix the same: 64 + 32 + 128 * 0.372 = 143.6 of them
        out["whole_model_estimate_s"] = round(dt * (96 + 128 * 4096.0 / 11008.0), 1)
        out["whole_model_note"] = ("extrapolated from the measured matrix, not run: the 224 Llama-7B-shaped "
                                   "matrices weighted by l")
    if args.cpu_baseline >= 2:
        ext = {}
        print("bench: oracle, q = 1", file=sys.stderr, flush=True)
        ext["q1_%dthreads" % threads] = _oracle_path(oracle, gi, m, n, r, p, 1, args.dtype, 7000)
        for (mm, nn) in ((4096, 4096), (11008, 4096)):
            print("bench: oracle, %dx%d" % (mm, nn), file=sys.stderr, flush=True)
            ext["%dx%d_%dthreads" % (mm, nn, threads)] = _oracle_path(oracle, gi, mm, nn, r, p, q, args.dtype, 7000)
        # one thread on the 1B-shaped gate/up matrix (2048x5461, r=512 p=16: an
        # eighth of the work of the matrix above), beside the same on all threads
        for nt in (threads, 1):
            print("bench: oracle, 2048x5461 on %d thread(s)" % nt, file=sys.stderr, flush=True)
            oracle.set_num_threads(nt)
            try:
                ext["2048x5461_r512_%dthread%s" % (nt, "s" if nt > 1 else "")] = _oracle_path(
                    oracle, gi, 2048, 5461, 512, 16, q, args.dtype, 7000)
            finally:
                oracle.set_num_threads(threads)
        if (m, n) == (4096, 11008):
            ext["whole_model_s_%dthreads" % threads] = round(
                64 * dt + 32 * ext["11008x4096_%dthreads" % threads]["total_s"]
                + 128 * ext["4096x4096_%dthreads" % threads]["total_s"], 1)
        ext["note"] = ("same spectrum, storage and r, p; whole_model = 64 x 4096x11008 + 32 x 11008x4096 + "
                       "128 x 4096x4096 of the measured per-matrix times")
        out["extended"] = ext
    return out


def time_configs(gl, gi, torch, dev):
    """The other workloads of the family, each on one stream (a second stream
    of this process for the small SVD's halves) and timed with HIP events
    around the library's calls only (gradient generation is outside them):
      single-256x688  one fp32 gradient, 1 subspace update + 1 projected Adam step
      llama-60m       56 fp32 gradients; 1 update, then 200 projected Adam steps,
                      each with fresh noise on the same planted singular vectors
      llama-350m      168 fp32 gradients; 600 steps of the scheduled step with an
                      update every T = 200 steps (Alg. 1; fixed gradients)
      llama-1b        168 bf16 gradients; one batched update of all, then one
                      projected Adam sweep (projection, Adam, weight update)"""
    st = torch.cuda.current_stream()
    aux = torch.cuda.Stream()
    mk = lambda: torch.cuda.Event(enable_timing=True)
    b1, b2, eps, lr, al = 0.9, 0.999, 1e-8, 1e-3, 0.25

    def groups(w, noise):
        out = []
        for gidx, (label, m, n, count) in enumerate(w.groups):
            s, l = min(m, n), max(m, n)
            G = gi.torch_planted_group(m, n, count, w.spectrum(s), noise, seed=8000 + 17 * gidx, dtype=w.dtype)
            out.append(dict(label=label, m=m, n=n, count=count, s=s, l=l, G=G,
                            W=torch.zeros((count, m, n), dtype=torch.float32, device=dev),
                            P=torch.empty((count, s, w.r), dtype=torch.float32, device=dev),
                            R=torch.empty((count, w.r, l), dtype=torch.float32, device=dev),
                            M=torch.zeros((count, w.r, l), dtype=torch.float32, device=dev),
                            V=torch.zeros((count, w.r, l), dtype=torch.float32, device=dev),
                            info=torch.zeros((count,), dtype=torch.int32, device=dev)))
            workspaces(out[-1], w)
        return out

    def workspaces(g, w):
        dt = g["G"].dtype
        g["ws"] = torch.empty((gl.galore_rsvd_workspace_size(g["m"], g["n"], w.r, w.p, g["count"], dt),),
                              dtype=torch.uint8, device=dev)
        pw = gl.galore_project_workspace_size(g["m"], g["n"], w.r, g["count"], dt)
        g["pws"] = torch.empty((pw,), dtype=torch.uint8, device=dev) if pw > 0 else False
        g["bws"] = torch.empty((gl.galore_project_back_workspace_size(g["m"], g["n"], w.r, g["count"]),),
                               dtype=torch.uint8, device=dev)

    def update_all(grs, w, idx):
        for g in grs:
            gl.galore_rsvd_update(g["G"], w.r, w.p, w.q, gi.sketch_seed(idx), 0, P=g["P"], info=g["info"],
                                  workspace=g["ws"], stream=st, aux_stream=aux)

    def adam_all(grs, t):
        for g in grs:
            gl.galore_project(g["P"], g["G"], R=g["R"], workspace=g["pws"], stream=st)
            gl.galore_lowrank_adam_step(g["R"], g["M"], g["V"], g["R"], b1, b2, eps, t, stream=st)
            gl.galore_project_back(g["P"], g["R"], g["W"], lr, al, workspace=g["bws"], stream=st)

    def check(grs):
        if any(int((g["info"] != 0).sum()) for g in grs):
            raise RuntimeError("small SVD did not converge")

    def timed(fn):
        e0, e1 = mk(), mk()
        e0.record(st)
        fn()
        e1.record(st)
        return e0, e1

    out = {}
    # single 256 x 688 gradient
    w = gi.WORKLOADS["single-256x688"]
    grs = [dict(label="single", m=256, n=688, count=1, s=256, l=688,
                G=torch.from_numpy(gi.store(gi.planted_gradient(256, 688, w.spectrum(256), w.noise, seed=1000),
                                            "f32").data).to(dev).unsqueeze(0))]
    g = grs[0]
    g.update(W=torch.zeros((1, 256, 688), device=dev), P=torch.empty((1, 256, w.r), device=dev),
             R=torch.empty((1, w.r, 688), device=dev), M=torch.zeros((1, w.r, 688), device=dev),
             V=torch.zeros((1, w.r, 688), device=dev), info=torch.zeros((1,), dtype=torch.int32, device=dev))
    workspaces(g, w)
    for _ in range(2):       # the second pass is timed
        u = timed(lambda: update_all(grs, w, 0))
        a = timed(lambda: adam_all(grs, 1))
    torch.cuda.synchronize()
    check(grs)
    out["single_256x688"] = {"update_ms": round(u[0].elapsed_time(u[1]), 4),
                             "adam_step_ms": round(a[0].elapsed_time(a[1]), 4),
                             "note": "one fp32 gradient, r=32 p=8 q=2: one subspace update, then one projected "
                                     "Adam step (projection, Adam, weight update); launch-bound"}
    del grs, g
    # Llama-60M-shaped: 1 update, then 200 steps with fresh noise
    w = gi.WORKLOADS["llama-60m"]
    grs = groups(w, 0.0)          # the noiseless planted part; noise drawn per step
    for g in grs:
        g["base"] = g["G"].clone()
    gen = torch.Generator(device=dev)
    gen.manual_seed(8100)

    def fresh():
        for g in grs:
            g["G"].copy_(g["base"])
            g["G"].add_(torch.randn(g["G"].shape, generator=gen, device=dev), alpha=w.noise)
    fresh()
    update_all(grs, w, 0)          # warm-up of the shapes
    torch.cuda.synchronize()
    fresh()
    u = timed(lambda: update_all(grs, w, 1))
    steps = []
    for t in range(1, 201):
        fresh()
        steps.append(timed(lambda: adam_all(grs, t)))
    torch.cuda.synchronize()
    check(grs)
    um = u[0].elapsed_time(u[1])
    sm = [a.elapsed_time(b) for a, b in steps]
    n60 = sum(g["count"] for g in grs)
    out["llama_60m"] = {"matrices": n60, "update_ms": round(um, 3), "updates_per_s": round(n60 / (um * 1e-3), 1),
                        "adam_step_ms_mean": round(sum(sm) / len(sm), 4), "run_200_steps_ms": round(um + sum(sm), 2),
                        "note": "56 fp32 gradients (8 layers x q,k,v,o 512x512, gate,up 512x1376, down 1376x512), "
                                "0.9^i + 1e-4 noise, r=128 p=8 q=2: one subspace update, then 200 projected Adam "
                                "steps with fresh noise on the same planted singular vectors"}
    del grs
    torch.cuda.empty_cache()
    # Llama-350M-shaped: 600 scheduled steps, update every 200
    w = gi.WORKLOADS["llama-350m"]
    grs = groups(w, w.noise)
    T = 200
    for g in grs:
        g["sws"] = torch.empty((gl.galore_step_workspace_size(g["m"], g["n"], w.r, w.p, g["count"], g["G"].dtype, 0),),
                               dtype=torch.uint8, device=dev)

    def step_all(tau):
        for g in grs:
            gl.galore_step(g["G"], g["W"], g["P"], g["M"], g["V"], w.r, w.p, w.q, gi.sketch_seed(tau // T), tau, T,
                           beta1=b1, beta2=b2, eps=eps, lr=lr, alpha=al, flags=0, info=g["info"], workspace=g["sws"],
                           stream=st, aux_stream=aux)
    step_all(0)                    # warm-up of the shapes
    torch.cuda.synchronize()
    for g in grs:
        g["M"].zero_()
        g["V"].zero_()
    evs = [timed(lambda tau=tau: step_all(tau)) for tau in range(600)]
    torch.cuda.synchronize()
    check(grs)
    ms = [a.elapsed_time(b) for a, b in evs]
    upd = [x for tau, x in enumerate(ms) if tau % T == 0]
    plain = [x for tau, x in enumerate(ms) if tau % T != 0]
    n350 = sum(g["count"] for g in grs)
    out["llama_350m"] = {"matrices": n350, "steps": 600, "T": T, "run_ms": round(sum(ms), 2),
                         "update_step_ms_mean": round(sum(upd) / len(upd), 3),
                         "plain_step_ms_mean": round(sum(plain) / len(plain), 4),
                         "note": "168 fp32 gradients (24 layers x q,k,v,o 1024x1024, gate,up 1024x2736, down "
                                 "2736x1024), (i+1)^-1 + 1e-4 noise, r=256 p=16 q=2: 600 calls of the scheduled "
                                 "step (Alg. 1: a subspace update when tau mod 200 = 0, projection, Adam and weight "
                                 "update every step; the same gradients each step)"}
    del grs, evs
    torch.cuda.empty_cache()
    # Llama-1B-shaped: one batched update of all 168, then one sweep
    w = gi.WORKLOADS["llama-1b"]
    grs = groups(w, w.noise)
    update_all(grs, w, 0)          # warm-up of the shapes
    adam_all(grs, 1)
    torch.cuda.synchronize()
    u = timed(lambda: update_all(grs, w, 1))
    a = timed(lambda: adam_all(grs, 2))
    torch.cuda.synchronize()
    check(grs)
    um, am = u[0].elapsed_time(u[1]), a[0].elapsed_time(a[1])
    n1b = sum(g["count"] for g in grs)
    out["llama_1b"] = {"matrices": n1b, "update_ms": round(um, 2), "updates_per_s": round(n1b / (um * 1e-3), 1),
                       "sweep_ms": round(am, 3),
                       "note": "168 bf16 gradients (24 layers x q,k,v,o 2048x2048, gate,up 2048x5461, down "
                               "5461x2048), (i+1)^-0.8 + 1e-4 noise, r=512 p=16 q=2: one subspace update of all, "
                               "then one projected Adam sweep over all"}
    del grs
    torch.cuda.empty_cache()
    return out


def main():
    args = parse()
    if args.write_traffic:
        write_traffic(args)
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py runs on exactly one GPU: the hot path is measured on one GPU's share "
              "(one process, no collectives); --gpus %d is not supported" % args.gpus, file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import galore_inputs as gi
    import paper_2504_20437_amd as gl

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    m, n, B, r, p, q = args.m, args.n, args.batch, args.r, args.p, args.q
    s, l = min(m, n), max(m, n)
    k = min(r + p, s)

    if args.copy_probe_mib > 0:
        src = torch.ones((args.copy_probe_mib, 1 << 18), dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        print("bench: copy probe of %d MiB done" % args.copy_probe_mib, file=sys.stderr, flush=True)
        del src, dst
    print("bench: generating %d x %dx%d %s gradients" % (B, m, n, args.dtype), file=sys.stderr, flush=True)
    G = gi.torch_planted_group(m, n, B, gi.spectrum_power(s, 0.7), 1e-4, seed=5000, dtype=args.dtype)
    gen = torch.Generator(device=dev)
    gen.manual_seed(5001)
    W = torch.empty((B, m, n), dtype=torch.float32, device=dev)
    for i in range(B):
        W[i].normal_(0.0, 0.02, generator=gen)
    P = torch.empty((B, s, r), dtype=torch.float32, device=dev)
    sigma = torch.empty((B, r), dtype=torch.float32, device=dev)
    info = torch.empty((B,), dtype=torch.int32, device=dev)
    R = torch.empty((B, r, l), dtype=torch.float32, device=dev)
    M = torch.zeros_like(R)
    V = torch.zeros_like(R)
    N = torch.empty_like(R)
    S = args.streams
    if S < 1 or B % S:
        raise SystemExit("--streams must divide the batch")
    C = B // S     # matrices per chunk
    chunks = []
    for ci in range(S):
        sl = slice(ci * C, (ci + 1) * C)
        pws_bytes = gl.galore_project_workspace_size(m, n, r, C, G.dtype)
        chunks.append(dict(
            sl=sl, stream=torch.cuda.current_stream() if ci == 0 else torch.cuda.Stream(),
            aux=torch.cuda.Stream(),     # second stream for the latency-bound stages (default priority)
            ws=torch.empty((gl.galore_rsvd_workspace_size(m, n, r, p, C, G.dtype),), dtype=torch.uint8, device=dev),
            pws=torch.empty((pws_bytes,), dtype=torch.uint8, device=dev) if pws_bytes > 0 else False,
            bws=torch.empty((gl.galore_project_back_workspace_size(m, n, r, C),), dtype=torch.uint8, device=dev)))
    torch.cuda.synchronize()
    stream = chunks[0]["stream"]      # stage events are recorded on chunk 0's stream
    aux0 = chunks[0]["aux"]
    outer = ("rsvd", "project", "adam", "project_back")
    cap = 96   # stage instances recorded per subspace update

    def run_chunk(ch, t, ev=None, sev=None):
        st, sl = ch["stream"], ch["sl"]
        if ev is not None:
            ev[0].record(st)
        if sev is None:
            gl.galore_rsvd_update(G[sl], r, p, q, gi.sketch_seed(t), sl.start, P=P[sl], sigma=sigma[sl], info=info[sl],
                                  workspace=ch["ws"], stream=st, aux_stream=ch["aux"])
            stages = None
        else:
            _, _, _, stages = gl.galore_rsvd_update_traced(G[sl], r, p, q, gi.sketch_seed(t), sev, sl.start, P=P[sl],
                                                           sigma=sigma[sl], info=info[sl], workspace=ch["ws"],
                                                           stream=st, aux_stream=ch["aux"])
        if ev is not None:
            ev[1].record(st)
        gl.galore_project(P[sl], G[sl], R=R[sl], workspace=ch["pws"], stream=st)
        if ev is not None:
            ev[2].record(st)
        gl.galore_lowrank_adam_step(R[sl], M[sl], V[sl], N[sl], 0.9, 0.999, 1e-8, t + 1, stream=st)
        if ev is not None:
            ev[3].record(st)
        gl.galore_project_back(P[sl], N[sl], W[sl], 1e-3, 0.25, workspace=ch["bws"], stream=st)
        if ev is not None:
            ev[4].record(st)
        return stages

    def step(t, ev=None, sev=None):
        if S > 1:                      # every chunk starts after the previous step's work on all streams
            mark = torch.cuda.Event()
            mark.record(stream)
            for ch in chunks[1:]:
                ch["stream"].wait_event(mark)
        stages = run_chunk(chunks[0], t, ev, sev)
        for ch in chunks[1:]:
            run_chunk(ch, t)
        if S > 1:                      # and chunk 0's stream waits for all of them
            for ch in chunks[1:]:
                done = torch.cuda.Event()
                done.record(ch["stream"])
                stream.wait_event(done)
        return stages

    for w in range(args.warmup):
        step(w)
        torch.cuda.synchronize()
        print("bench: warmup %d done" % w, file=sys.stderr, flush=True)
    if args.warmup > 0 and int((info != 0).sum()) != 0:
        raise RuntimeError("small SVD did not converge for %d matrices" % int((info != 0).sum()))

    mk = lambda: torch.cuda.Event(enable_timing=True)
    events = [[mk() for _ in range(5)] for _ in range(args.steps)]
    sevents = [[mk() for _ in range(2 * cap)] for _ in range(args.steps)]
    for evs in sevents:
        for e in evs:
            e.record(stream)     # torch creates the HIP event on its first record
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    stage_lists = []
    for i in range(args.steps):
        stage_lists.append(step(args.warmup + i, events[i], sevents[i]))
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    bad = int((info != 0).sum())
    if bad:
        raise RuntimeError("small SVD did not converge for %d matrices" % bad)

    # ---- per-stage times (ms per step) and per-launch durations ---------------
    per_stage = {st: 0.0 for st in outer}
    sub = {}
    launches = {}    # single-launch kernel class -> list of durations (ms)
    for ev, sev, stl in zip(events, sevents, stage_lists):
        for j, st in enumerate(outer):
            d = ev[j].elapsed_time(ev[j + 1])
            per_stage[st] += d
            if st != "rsvd":
                launches.setdefault(st, []).append(d)
        first_a = True
        for i, name in enumerate(stl):
            d = sev[2 * i].elapsed_time(sev[2 * i + 1])
            sub[name] = sub.get(name, 0.0) + d
            # with a bf16 gradient the first A product takes the bf16-valued sketch
            # as one exact plane: a different launch shape, timed on its own
            key = name
            if name == "product_A" and first_a:
                first_a = False
                if args.dtype == "bf16":
                    key = "product_A_sketch"
            launches.setdefault(key, []).append(d)
    per_stage = {st: v / args.steps for st, v in per_stage.items()}
    sub = {st: v / args.steps for st, v in sub.items()}
    ms_per_step = wall * 1000.0 / args.steps

    # algorithmic work of one launch of each single-launch kernel class
    # (flops, except bytes for Adam), for one chunk (the launches timed are
    # chunk 0's)
    n_gram_s = (2 if q == 0 else q + 2)          # Grams of s x k blocks per update
    n_gram_l = q + 1                              # Grams of l x k blocks per update
    # products with a bf16-stored G run on the bf16 matrix cores as three exact
    # bf16 products per fp32-accurate one (bf16x3.hip): bf16 peak, 3 MFMA flops
    # per algorithmic flop
    prod_bound = "mfma_bf16x3" if args.dtype == "bf16" else "mfma"
    work = {
        "product_A": (prod_bound, 2.0 * s * l * k * C),
        "product_A_sketch": ("mfma_bf16" if args.dtype == "bf16" else "mfma", 2.0 * s * l * k * C),
        "product_At": (prod_bound, 2.0 * s * l * k * C),
        "projector": ("mfma", 2.0 * s * k * r * C),
        "project": (prod_bound, 2.0 * r * s * l * C),
        "project_back": ("mfma_bf16x6", 2.0 * r * s * l * C),
        "adam": ("hbm", float(ADAM_BYTES_PER_ELEM * C * r * l)),
        # symmetric Gram X^T X: rows * k * (k + 1) flops, averaged over its launches;
        # exact on the int8 matrix cores as nine digit-plane products (gram_i8.hip)
        "gram": ("mfma_i8x9", (n_gram_s * s + n_gram_l * l) * k * (k + 1.0) * C / (n_gram_s + n_gram_l)),
        # Q = Y R^-1 with triangular R^-1: rows * k * (k + 1) flops, averaged
        "triangular": ("mfma", ((n_gram_s * s + (n_gram_l - 1) * l) * k * (k + 1.0) * C
                                / max(1, n_gram_s + n_gram_l - 1))),
    }
    work["products"] = work["product_A"]          # both products run the same kernel on the same work
    for cls, (members, _, _) in KERNEL_CLASSES.items():
        durs_c = [d for mname in members for d in launches.get(mname, [])]
        if durs_c:
            launches.setdefault(cls, durs_c)
    kern = args.roofline_kernel
    if kern == "auto":
        cand = [c for c in KERNEL_CLASSES if c in launches]
        kern = max(cand, key=lambda c: sum(launches[c]))
    durs = launches[kern]
    avg_ms = sum(durs) / len(durs)
    bound, units = work[kern]
    traffic = None
    traffic_note = "no counter reading for this kernel and workload"
    try:
        with open(args.traffic_json) as f:
            rec = json.load(f).get(workload_key(kern, args))
        if rec is not None:
            if rec.get("source_sha256") == source_hash(kernel_class(kern, args.dtype)[2]):
                traffic = rec["bytes_per_launch"]
                traffic_note = "rocprofv3 FETCH_SIZE x %.3g + WRITE_SIZE x %.3g per launch" % (
                    rec["fetch_factor"], rec["write_factor"])
            else:
                traffic_note = "counter reading is of an earlier version of the kernel"
    except (OSError, ValueError):
        pass
    if bound == "hbm":
        ach = units / (avg_ms * 1e-3) / 1e9
        roof = {"kernel": kern, "bound": "hbm", "achieved": round(ach, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(ach / HBM_PEAK_GBS, 4), "traffic": traffic}
    else:
        peak = {"mfma": FP32_MFMA_PEAK_TFS, "mfma64": FP64_MFMA_PEAK_TFS, "mfma_bf16x3": BF16_MFMA_PEAK_TFS,
                "mfma_bf16": BF16_MFMA_PEAK_TFS,
                "mfma_bf16x6": BF16_MFMA_PEAK_TFS, "mfma_i8x9": INT8_MFMA_PEAK_TOPS}[bound]
        ach = units / (avg_ms * 1e-3) / 1e12
        roof = {"kernel": kern, "bound": "mfma", "achieved": round(ach, 2), "peak": peak, "unit": "TFLOP/s",
                "frac": round(ach / peak, 4), "traffic": traffic}
        if bound == "mfma_bf16x3":
            roof["mfma_dtype"] = "bf16 (3 exact bf16 products per fp32-accurate product)"
            roof["frac_of_3x_ceiling"] = round(3.0 * ach / peak, 4)
            # the same fp32-accurate product on the fp32 matrix cores would be
            # capped at their dense peak
            roof["vs_fp32_mfma_peak"] = {"peak": FP32_MFMA_PEAK_TFS, "frac": round(ach / FP32_MFMA_PEAK_TFS, 4)}
        if bound == "mfma_i8x9":
            roof["mfma_dtype"] = "int8 (9 exact digit-plane products per fp32-input Gram entry)"
            roof["frac_of_9x_ceiling"] = round(9.0 * ach / peak, 4)
        if bound == "mfma_bf16x6":
            roof["mfma_dtype"] = "bf16 (6 bf16 plane products per fp32-accurate product)"
            roof["frac_of_6x_ceiling"] = round(6.0 * ach / peak, 4)
    roof["traffic_note"] = traffic_note
    roof["launches_timed"] = len(durs)
    roof["avg_launch_ms"] = round(avg_ms, 3)
    roof["work_per_launch"] = units
    adam_gbs = work["adam"][1] / (per_stage["adam"] * 1e-3) / 1e9
    rates = {}
    for c, (bd, units_c) in work.items():
        if c in launches:
            a = sum(launches[c]) / len(launches[c])
            rates[c] = round(units_c / (a * 1e-3) / (1e9 if bd == "hbm" else 1e12), 2)

    # the chip's own peaks under load: sustained bf16 matrix-core rate (probe
    # kernel, register operands only) and device-to-device copy bandwidth
    sink = torch.empty((2048 * 256,), dtype=torch.float32, device=dev)
    pe = [mk() for _ in range(4)]
    for j in range(2):
        pe[2 * j].record(stream)
        probe_flops = gl.galore_probe_mfma_bf16(2000, 2048, sink, stream=stream)
        pe[2 * j + 1].record(stream)
    torch.cuda.synchronize()
    mfma_meas = probe_flops / (pe[2].elapsed_time(pe[3]) * 1e-3) / 1e12
    csrc_t = torch.empty((1 << 28,), dtype=torch.float32, device=dev)
    cdst_t = torch.empty_like(csrc_t)
    ce = [mk() for _ in range(4)]
    for j in range(2):
        ce[2 * j].record(stream)
        gl.galore_probe_copy(csrc_t, cdst_t, stream=stream)
        ce[2 * j + 1].record(stream)
    torch.cuda.synchronize()
    hbm_meas = 2.0 * csrc_t.numel() * 4 / (ce[2].elapsed_time(ce[3]) * 1e-3) / 1e9
    del sink, csrc_t, cdst_t
    measured_peaks = {"bf16_mfma_tflops": round(mfma_meas, 1), "hbm_copy_gbs": round(hbm_meas, 1),
                      "note": "sustained bf16 MFMA rate of a register-only probe kernel (2048 workgroups); "
                              "streaming copy probe of 1 GiB, one 16-byte vector per thread (bytes read + written)"}
    if roof["bound"] == "hbm":
        roof["peak_measured"] = measured_peaks["hbm_copy_gbs"]
    elif roof.get("mfma_dtype", "").startswith("bf16"):
        roof["peak_measured"] = measured_peaks["bf16_mfma_tflops"]
    if "peak_measured" in roof:
        roof["frac_measured"] = round(roof["achieved"] / roof["peak_measured"], 4)

    switch_ms = upd_ms = plain_ms = None
    lowbit, exact_svd, whole_model, adam8 = {}, None, None, None
    T_sched = 200
    if args.extras:
        # subspace switch (once per T steps): signs of a new projector matched to
        # the previous one and the first moment re-expressed in the new basis;
        # timed outside the step on a copy of the current projector
        P_new = P.clone()
        M_sw = torch.empty_like(M)
        aws = torch.empty((gl.galore_align_workspace_size(r, B),), dtype=torch.uint8, device=dev)
        sw = [mk() for _ in range(4)]
        for j in range(2):
            sw[2 * j].record(stream)
            gl.galore_align_projector(P, P_new, M, M_out=M_sw, workspace=aws, stream=stream)
            sw[2 * j + 1].record(stream)
        torch.cuda.synchronize()
        switch_ms = sw[2].elapsed_time(sw[3])
        del P_new, M_sw, aws

        # the schedule through the one-call step: a window of steps tau = T .. T+9
        # (an update step with the switch, then nine steps on the same projector)
        T_sched = 200
        sws = torch.empty((gl.galore_step_workspace_size(m, n, r, p, B, G.dtype, 3),), dtype=torch.uint8, device=dev)
        sinfo = torch.zeros((B,), dtype=torch.int32, device=dev)
        win = [mk() for _ in range(11)]
        win[0].record(stream)
        for j in range(10):
            gl.galore_step(G, W, P, M, V, r, p, q, gi.sketch_seed(1), T_sched + j, T_sched, flags=3, info=sinfo,
                           workspace=sws, stream=stream, aux_stream=aux0)
            win[j + 1].record(stream)
        torch.cuda.synchronize()
        if int((sinfo != 0).sum()):
            raise RuntimeError("small SVD did not converge in the scheduled step")
        upd_ms = win[0].elapsed_time(win[1])
        plain_ms = win[1].elapsed_time(win[10]) / 9.0
        del sws

        # low-bit projector: quantise the batch's projectors once per update, then
        # each step projects and back-projects with the codes
        lowbit = {}
        for bits in (8, 4):
            qws = torch.empty((gl.galore_project_quantized_workspace_size(m, n, r, B),), dtype=torch.uint8, device=dev)
            qbws = torch.empty((gl.galore_project_back_quantized_workspace_size(m, n, r, B),), dtype=torch.uint8,
                               device=dev)
            qe = [mk() for _ in range(8)]
            for j in range(2):       # the second pass is timed
                qe[0].record(stream)
                Pq = gl.galore_quantize_projector(P, bits, stream=stream)
                qe[1].record(stream)
                gl.galore_project_quantized(Pq, G, R=R, workspace=qws, stream=stream)
                qe[2].record(stream)
                gl.galore_lowrank_adam_step(R, M, V, N, 0.9, 0.999, 1e-8, 2, stream=stream)
                qe[3].record(stream)
                gl.galore_project_back_quantized(Pq, N, W, 1e-3, 0.25, workspace=qbws, stream=stream)
                qe[4].record(stream)
            torch.cuda.synchronize()
            lowbit["int%d" % bits] = {
                "quantize_ms": round(qe[0].elapsed_time(qe[1]), 3),
                "project_ms": round(qe[1].elapsed_time(qe[2]), 3),
                "adam_ms": round(qe[2].elapsed_time(qe[3]), 3),
                "project_back_ms": round(qe[3].elapsed_time(qe[4]), 3),
                "step_ms": round(qe[1].elapsed_time(qe[4]), 3),
                "projector_bytes": int(Pq.codes.numel() + 4 * Pq.scales.numel()),
            }
            del qws, qbws, Pq

        # exact SVD (k = s) against the randomized one on the same 8 matrices
        if s <= 4096:
            Bx = min(B, 8)
            xws = torch.empty((gl.galore_svd_workspace_size(m, n, r, Bx, G.dtype),), dtype=torch.uint8, device=dev)
            xe = [mk() for _ in range(8)]
            for j in range(2):
                xe[4 * j].record(stream)
                _, _, xinfo = gl.galore_svd_update(G[:Bx], r, workspace=xws, stream=stream, aux_stream=aux0)
                xe[4 * j + 1].record(stream)
                gl.galore_rsvd_update(G[:Bx], r, p, q, gi.sketch_seed(0), 0, P=P[:Bx], sigma=sigma[:Bx], info=info[:Bx],
                                      workspace=chunks[0]["ws"], stream=stream, aux_stream=aux0)
                xe[4 * j + 2].record(stream)
            torch.cuda.synchronize()
            if int((xinfo != 0).sum()):
                raise RuntimeError("exact SVD did not converge")
            x_ms, rs_ms = xe[4].elapsed_time(xe[5]), xe[5].elapsed_time(xe[6])
            exact_svd = {"batch": Bx, "exact_ms_per_matrix": round(x_ms / Bx, 3),
                         "rsvd_ms_per_matrix": round(rs_ms / Bx, 3), "speedup": round(x_ms / rs_ms, 2),
                         "note": "exact top-r SVD (sketch as wide as the short side, k = %d, no power iteration) against "
                                 "the randomized update (k = %d, q = %d) on the same %d matrices" % (s, k, q, Bx)}
            del xws
        else:
            exact_svd = None

        # the whole Llama-7B-shaped model on this GPU: 128 square (q, k, v, o),
        # 64 gate/up (the batch above) and 32 down matrices; a subspace update of
        # all 224 with q = 1 and with q = 2, and one projected Adam step over all
        whole_model = None
        if args.whole_model and (m, n, B, S) == (4096, 11008, 64, 1):
            groups = [{"name": "q,k,v,o 4096x4096", "m": 4096, "n": 4096, "count": 128, "seed": 5100},
                      {"name": "down 11008x4096", "m": 11008, "n": 4096, "count": 32, "seed": 5200}]
            for gr in groups:
                gm, gn, gc = gr["m"], gr["n"], gr["count"]
                gs, gl_ = min(gm, gn), max(gm, gn)
                print("bench: generating %d x %dx%d %s gradients" % (gc, gm, gn, args.dtype), file=sys.stderr, flush=True)
                gr["G"] = gi.torch_planted_group(gm, gn, gc, gi.spectrum_power(gs, 0.7), 1e-4, seed=gr["seed"],
                                                 dtype=args.dtype)
                gr["W"] = torch.zeros((gc, gm, gn), dtype=torch.float32, device=dev)
                gr["P"] = torch.empty((gc, gs, r), dtype=torch.float32, device=dev)
                gr["sigma"] = torch.empty((gc, r), dtype=torch.float32, device=dev)
                gr["info"] = torch.empty((gc,), dtype=torch.int32, device=dev)
                gr["R"] = torch.empty((gc, r, gl_), dtype=torch.float32, device=dev)
                gr["M"] = torch.zeros_like(gr["R"])
                gr["V"] = torch.zeros_like(gr["R"])
                gr["ws"] = torch.empty((gl.galore_rsvd_workspace_size(gm, gn, r, p, gc, G.dtype),), dtype=torch.uint8,
                                       device=dev)
                pw = gl.galore_project_workspace_size(gm, gn, r, gc, G.dtype)
                gr["pws"] = torch.empty((pw,), dtype=torch.uint8, device=dev) if pw > 0 else False
                gr["bws"] = torch.empty((gl.galore_project_back_workspace_size(gm, gn, r, gc),), dtype=torch.uint8,
                                        device=dev)
            groups.insert(1, {"name": "gate/up 4096x11008", "m": m, "n": n, "count": B, "G": G, "W": W, "P": P,
                              "sigma": sigma, "info": info, "R": R, "M": M, "V": V, "ws": chunks[0]["ws"],
                              "pws": chunks[0]["pws"], "bws": chunks[0]["bws"]})
            torch.cuda.synchronize()
            wm_ms = {}
            for qq in (1, 2):
                e0, e1 = mk(), mk()
                e0.record(stream)
                for gr in groups:
                    gl.galore_rsvd_update(gr["G"], r, p, qq, gi.sketch_seed(qq), 0, P=gr["P"], sigma=gr["sigma"],
                                          info=gr["info"], workspace=gr["ws"], stream=stream, aux_stream=aux0)
                e1.record(stream)
                torch.cuda.synchronize()
                wm_ms["update_q%d" % qq] = e0.elapsed_time(e1)
                if any(int((gr["info"] != 0).sum()) for gr in groups):
                    raise RuntimeError("small SVD did not converge in the whole-model update")
            e0, e1 = mk(), mk()
            e0.record(stream)
            for gr in groups:
                gl.galore_project(gr["P"], gr["G"], R=gr["R"], workspace=gr["pws"], stream=stream)
                gl.galore_lowrank_adam_step(gr["R"], gr["M"], gr["V"], gr["R"], 0.9, 0.999, 1e-8, 1, stream=stream)
                gl.galore_project_back(gr["P"], gr["R"], gr["W"], 1e-3, 0.25, workspace=gr["bws"], stream=stream)
            e1.record(stream)
            torch.cuda.synchronize()
            wm_ms["adam_step"] = e0.elapsed_time(e1)
            nmat = sum(gr["count"] for gr in groups)
            whole_model = {"matrices": nmat,
                           "update_q1_ms": round(wm_ms["update_q1"], 1), "update_q2_ms": round(wm_ms["update_q2"], 1),
                           "projected_adam_step_ms": round(wm_ms["adam_step"], 1),
                           "note": "Llama-7B-shaped model, all %d projection matrices on this GPU (128 x 4096x4096, "
                                   "64 x 4096x11008, 32 x 11008x4096, %s, r=%d p=%d): one subspace update of every "
                                   "matrix with q = 1 and with q = 2, and one projected Adam step (projection, Adam, "
                                   "weight update) over all" % (nmat, args.dtype, r, p)}
            for gr in groups:
                if gr["name"].startswith("gate"):
                    continue
                for key in ("G", "W", "P", "R", "M", "V", "ws", "pws", "bws"):
                    gr[key] = None
            torch.cuda.empty_cache()

        # 8-bit moments (E4M3 / E5M2 codes, one scale per 2048-element block)
        st8 = gl.Adam8State(r, l, B, device=dev)
        a8 = [mk() for _ in range(4)]
        for j in range(2):
            a8[2 * j].record(stream)
            gl.galore_lowrank_adam8_step(R, st8, N=N, beta1=0.9, beta2=0.999, eps=1e-8, t=j + 1, stream=stream)
            a8[2 * j + 1].record(stream)
        torch.cuda.synchronize()
        adam8_ms = a8[2].elapsed_time(a8[3])
        adam8 = {"ms": round(adam8_ms, 3), "hbm_gbs": round(12.0 * B * r * l / (adam8_ms * 1e-3) / 1e9, 1),
                 "state_bytes": int(2 * (st8.M8.numel() + 4 * st8.Ms.numel())),
                 "note": "8-bit block-wise Adam on the whole batch: 12 bytes per element (R, N fp32; M, V one byte each "
                         "in and out); fp32 moments take %d bytes" % (8 * B * r * l)}
        del st8

    out = {
        "metric": "rSVD subspace updates/sec at 4096x11008 r=1024; low-rank Adam step HBM GB/s",
        "value": round(B / (ms_per_step * 1e-3), 3),
        "unit": "updates/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32" if args.dtype == "f32" else "f32 (bf16-stored gradients)",
        "data": "synthetic",
        "config": {"workload": "Llama-7B-shaped gate/up gradients: %d x %dx%d %s, planted spectrum "
                               "(i+1)^-0.7 + 1e-4 noise, r=%d p=%d q=%d (k=%d)"
                               % (B, m, n, args.dtype, r, p, q, k),
                   "batch": B, "m": m, "n": n, "r": r, "p": p, "q": q, "streams": S},
        "adam_hbm_gbs": round(adam_gbs, 1),
        "stage_ms": {st: round(v, 3) for st, v in per_stage.items()},
        "stage_note": ("stage and kernel times are chunk 0's (%d matrices) on its stream, overlapping the other "
                       "%d chunk(s)" % (C, S - 1)) if S > 1 else "stage and kernel times of the whole batch",
        "rsvd_stage_ms": {st: round(v, 3) for st, v in sorted(sub.items(), key=lambda x: -x[1])},
        "kernel_rates": rates,
        "roofline": roof,
        "schedule": None if upd_ms is None else {
            "T": T_sched, "update_step_ms": round(upd_ms, 3), "plain_step_ms": round(plain_ms, 3),
            "amortised_step_ms": round((upd_ms + (T_sched - 1) * plain_ms) / T_sched, 3),
            "note": "galore_step on the whole batch: the update step (subspace update, switch with "
                    "re-expression, projection, Adam, back-projection) and the mean of the next nine"},
        "measured_peaks": measured_peaks,
        "whole_model": whole_model,
        "adam8": adam8,
        "exact_svd": exact_svd,
        "lowbit_projector": dict(lowbit, note="steps on a fixed projector with its int8 / int4 codes (whole batch): "
                                               "projection, Adam, back-projection; fp32 projector bytes %d"
                                               % (4 * B * s * r)) if lowbit else None,
        "switch_ms": None if switch_ms is None else round(switch_ms, 3),
        "switch_note": None if switch_ms is None else (
            "subspace switch of the whole batch (sign alignment + first-moment re-expression), "
            "once per T steps: %.4f ms per step at T=200" % (switch_ms / 200.0)),
    }
    del G, W, R, M, V, N, chunks
    torch.cuda.empty_cache()
    if args.configs:
        print("bench: timing the other workloads", file=sys.stderr, flush=True)
        out["configs"] = time_configs(gl, gi, torch, dev)
    if args.cpu_baseline:
        print("bench: timing the oracle on the host", file=sys.stderr, flush=True)
        out["cpu_baseline"] = cpu_baseline(args)
    else:
        out["cpu_baseline"] = None
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
