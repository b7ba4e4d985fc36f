"""Benchmark of the bucket-level resolve step on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]

A step is one pass of the whole hot path over the workload's gradients,
already resident in HBM: the per-bucket Gram matrices, the per-bucket solve
and the combined update.  The step runs what bkmoo_resolve runs for the
workload: its cooperative kernel (the pipelined, partly resident one) when
it takes that path, as one call, else the two-pass kernels through the three stage entry points in stream order
(identical results to bkmoo_resolve's two-pass path, and each stage can be
timed).  The default workload is the Llama-3-8B-shaped K=4 bf16 MGDA
(Frank-Wolfe, 20 iterations) case with 25 MiB buckets.  Prints ONE JSON
line.

Reported next to the throughput:
  roofline     the longest kernel of a step (HBM-bound), timed with HIP
               events on its launch stream inside the timed region:
               algorithmic bytes per launch / average launch duration,
               against MI355X's 8 TB/s.  A streaming pass counts the bytes
               it must move (Gram K*s*N, combine (K+1)*s*N); a cooperative
               kernel, which does the whole step, counts the one-read floor
               K*s*N + s_out*N and gets no credit for its re-reads, part of
               which the last-level cache serves (`requested_frac`: the
               bytes it does request, re-reads included, per launch
               duration, over 8 TB/s).  `traffic` (bytes per launch) comes
               from the committed rocprofv3 counter summary (FETCH_SIZE +
               WRITE_SIZE, scaled by a copy kernel's reading) when it
               matches the current kernel source, else null.  These counters
               sit between the L2 and the fabric: on gfx950 no counter
               separates Infinity Cache hits from DRAM, so for a kernel that
               re-reads (the cooperative one) `traffic` is an upper bound of
               its DRAM bytes and the one-read floor a lower bound
               (`traffic_kind`, `dram_bytes_bounds`);
  two_pass     when the step ran a cooperative kernel: the plain two-pass
               resolve on the same inputs, with its (2K+1)*s*N bytes;
  cpu_baseline the float64 oracle on a bounded prefix of the same buckets,
               one bucket per worker thread over this host's cores (count
               and model).
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
sys.path.insert(0, ROOT)

PEAK_HBM_GBPS = 8000.0
METRIC = "resolved grad elems/s (K·N/s) + achieved HBM GB/s vs peak, K=4 MGDA 8B-shape"
DEFAULT_WORKLOAD = "llama3-8b-k4-mgda-bf16"
PROFILE_DIR = os.path.join(ROOT, "profiles")


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


# The sources each timed kernel is compiled from (its file and the headers it
# includes): a committed counter summary applies while these are unchanged.
KERNEL_SOURCES = {
    "gram": ["gram.hip", "stream_common.h", "internal.h"],
    "combine": ["combine.hip", "combine_impl.h", "stream_common.h", "internal.h"],
    "hybrid": ["hybrid.hip", "coop_common.h", "combine_impl.h", "solve_impl.h", "stream_common.h",
               "internal.h"],
    "refill": ["refill.hip", "refill.h", "coop_common.h", "combine_impl.h", "solve_impl.h",
               "stream_common.h", "internal.h"],
}


def kernel_source_sha(kernel: str) -> str:
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2606_05613_amd", "csrc")
    for f in KERNEL_SOURCES[kernel]:
        with open(os.path.join(csrc, f), "rb") as fh:
            h.update(f.encode())
            h.update(fh.read())
    return h.hexdigest()[:16]


def committed_traffic(workload: str, kernel: str):
    """Bytes per launch of `kernel` on `workload` between the L2 and the
    fabric (FETCH_SIZE + WRITE_SIZE, calibrated) from the committed rocprofv3
    counter summary, if it was taken on the current source."""
    path = os.path.join(PROFILE_DIR, f"{kernel}_{workload}_pmc.md")
    if not os.path.exists(path):
        return None
    text = open(path).read()
    sha = re.search(r"source_sha:\s*(\w+)", text)
    val = re.search(r"fabric_bytes_per_launch:\s*([0-9.eE+]+)", text)
    if not sha or not val or sha.group(1) != kernel_source_sha(kernel):
        return None
    return float(val.group(1))


# worker threads of the CPU baseline: the host's cores, at most the 16 a
# one-GPU share of the machine has
CPU_WORKERS_MAX = 16


def cpu_baseline(wl, grads, target_s: float):
    """The oracle, as it stands, on a prefix of the workload's buckets: one
    bucket per worker thread (numpy releases the interpreter lock in its
    array work; its BLAS is held to one thread per worker), batches of one
    bucket per worker until about target_s of compute.  The device-to-host
    copies of a batch are not timed."""
    import concurrent.futures
    import numpy as np
    import oracle
    from synth import host_rows
    from threadpoolctl import threadpool_limits
    workers = max(1, min(os.cpu_count() or 1, CPU_WORKERS_MAX))
    offs = wl.offsets()
    orders = wl.orders() if wl.method == "pcgrad" else None

    def one(b, rows):
        lo, hi = int(offs[b]), int(offs[b + 1])
        oracle.resolve(rows, np.array([0, hi - lo]), wl.method, max_iter=wl.max_iter,
                       cagrad_c=wl.cagrad_c, orders=None if orders is None else orders[b:b + 1])

    done_elems, spent, nb = 0, 0.0, 0
    with threadpool_limits(limits=1), concurrent.futures.ThreadPoolExecutor(workers) as ex:
        while nb < wl.B and spent < target_s:
            batch = list(range(nb, min(wl.B, nb + workers)))
            rows = [host_rows(grads, int(offs[b]), int(offs[b + 1])) for b in batch]   # not timed
            t0 = time.perf_counter()
            list(ex.map(one, batch, rows))
            spent += time.perf_counter() - t0
            done_elems += sum(int(offs[b + 1] - offs[b]) for b in batch)
            nb = batch[-1] + 1
            del rows
    cores = workers
    cpu = ""
    try:
        with open("/proc/cpuinfo") as fh:
            cpu = next((ln.split(":", 1)[1].strip() for ln in fh if ln.startswith("model name")), "")
    except OSError:
        pass
    return {"value": wl.K * done_elems / spent, "unit": "elem/s", "cores": int(cores), "cpu": cpu,
            "host_cpus": os.cpu_count(), "kind": "oracle",
            "sample": f"first {nb} of {wl.B} buckets ({wl.K}x{done_elems} elements), oracle.resolve "
                      f"end to end (Gram, {wl.method}, combine, rounding), one bucket per thread on "
                      f"{cores} threads, {spent:.1f} s"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD)
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--path", choices=["auto", "two-pass", "hybrid", "refill"], default="auto",
                    help="force bkmoo_resolve's implementation (default: the library's choice)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="first run one plain elementwise kernel that reads 2 GiB and writes "
                         "2 GiB (a known-size reference for rocprofv3 FETCH_SIZE / WRITE_SIZE)")
    args = ap.parse_args()

    if args.gpus != 1:
        print(f"bench.py measures one GPU only (got --gpus {args.gpus}): the library has no multi-GPU "
              "path (the bucket-level resolve would shard by buckets and bucket slices; not "
              "implemented).", flush=True)
        sys.exit(2)

    import torch
    from paper_2606_05613_amd import bkmoo
    from synth import WORKLOADS, fill_grads

    wl = WORKLOADS[args.workload]
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    K, N, B, s = wl.K, wl.N, wl.B, wl.elem_bytes
    log(f"workload {wl.name}: K={K} N={N} B={B} {wl.dtype} {wl.method}; generating "
        f"{K * N * s / 1e9:.1f} GB of gradients on {torch.cuda.get_device_name(dev)}")
    t0 = time.time()
    last = [t0]

    def progress(b):
        if time.time() - last[0] > 5:
            last[0] = time.time()
            log(f"  generated bucket {b + 1}/{B}")

    if args.copy_calibration:
        src = torch.ones(1 << 30, dtype=torch.bfloat16, device=dev)     # 2 GiB
        flush = torch.zeros(1 << 31, dtype=torch.uint8, device=dev)     # evicts L2 and Infinity Cache
        dst = torch.mul(src, 2.0)                                        # reads 2 GiB, writes 2 GiB
        torch.cuda.synchronize()
        log("copy calibration: elementwise kernel, 2 GiB read + 2 GiB written")
        del src, dst, flush
    grads = fill_grads(wl, device=dev, progress=progress)
    torch.cuda.synchronize()
    log(f"generated in {time.time() - t0:.1f} s")
    offs = torch.from_numpy(wl.offsets()).to(dev)
    order = torch.from_numpy(wl.orders()).to(dev) if wl.method == "pcgrad" else None
    out = torch.empty(N, dtype=grads.dtype, device=dev)
    ws = torch.empty(bkmoo.workspace_size(K, N, B, wl.dtype), dtype=torch.uint8, device=dev)
    G = torch.empty((B, K, K), dtype=torch.float64, device=dev)
    W = torch.empty((B, K), dtype=torch.float32, device=dev)
    A = torch.empty((B, K), dtype=torch.float64, device=dev)
    stream = torch.cuda.current_stream(dev)
    forced = {"auto": 0, "two-pass": bkmoo.PATH_TWO_PASS, "hybrid": bkmoo.PATH_HYBRID,
              "refill": bkmoo.PATH_REFILL}[args.path]
    bkmoo.set_resolve_path(forced)
    path = bkmoo.resolve_path(grads, B + 1, wl.method, wl.max_iter)
    path_name = {bkmoo.PATH_TWO_PASS: "two-pass", bkmoo.PATH_HYBRID: "hybrid", bkmoo.PATH_REFILL: "refill"}[path]
    # the cooperative path is one kernel: time the whole resolve call
    cooperative = path in (bkmoo.PATH_HYBRID, bkmoo.PATH_REFILL)
    traffic_bytes = bkmoo.resolve_traffic(K, wl.offsets(), wl.dtype, path, method=wl.method, max_iter=wl.max_iter)
    log(f"resolve path: {path_name}; it requests {traffic_bytes / 1e9:.2f} GB from memory per step")

    def step(ev=None):
        if cooperative:
            if ev is not None:
                ev[0].record(stream)
            bkmoo.resolve(grads, offs, wl.method, wl.max_iter, wl.cagrad_c, pcgrad_order=order, out=out,
                          gram_out=G, weights=W, aux=A, workspace=ws)
            if ev is not None:
                ev[3].record(stream)
            return
        if ev is not None:
            ev[0].record(stream)
        bkmoo.gram(grads, offs, gram_out=G, workspace=ws)
        if ev is not None:
            ev[1].record(stream)
        bkmoo.solve(G, wl.method, wl.max_iter, wl.cagrad_c, pcgrad_order=order, weights=W, aux=A)
        if ev is not None:
            ev[2].record(stream)
        bkmoo.combine(grads, offs, W, out=out, workspace=ws)
        if ev is not None:
            ev[3].record(stream)

    for i in range(args.warmup):
        step()
    torch.cuda.synchronize()
    if bkmoo.read_device_error(ws) != 0:
        raise RuntimeError(f"device error word 0x{bkmoo.read_device_error(ws):x} after the warmup")
    log(f"warmup done ({args.warmup} steps); timing {args.steps} steps")

    events = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    for i in range(args.steps):
        step(events[i])
    torch.cuda.synchronize()
    t_wall = time.perf_counter() - t_start
    ms_step = t_wall * 1e3 / args.steps
    if cooperative:
        st = {"resolve": sum(ev[0].elapsed_time(ev[3]) for ev in events) / args.steps}
    else:
        st = {"gram": 0.0, "solve": 0.0, "combine": 0.0}
        for ev in events:
            st["gram"] += ev[0].elapsed_time(ev[1]) / args.steps
            st["solve"] += ev[1].elapsed_time(ev[2]) / args.steps
            st["combine"] += ev[2].elapsed_time(ev[3]) / args.steps
    if bkmoo.read_device_error(ws) != 0:
        raise RuntimeError(f"device error word 0x{bkmoo.read_device_error(ws):x} after the timed steps")
    log(f"{ms_step:.3f} ms/step; stages (ms) " + ", ".join(f"{k} {v:.3f}" for k, v in st.items()))

    # the plain two-pass resolve on the same inputs, reported beside a
    # cooperative path's figure (whose re-reads may hit the last-level cache)
    two_pass = None
    if cooperative:
        bkmoo.set_resolve_path(bkmoo.PATH_TWO_PASS)
        try:
            def two_pass_step():
                bkmoo.resolve(grads, offs, wl.method, wl.max_iter, wl.cagrad_c, pcgrad_order=order, out=out,
                              gram_out=G, weights=W, aux=A, workspace=ws)
            for _ in range(2):
                two_pass_step()
            e0t, e1t = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            reps = max(3, args.steps // 2)
            e0t.record(stream)
            for _ in range(reps):
                two_pass_step()
            e1t.record(stream)
            torch.cuda.synchronize()
        finally:
            bkmoo.set_resolve_path(forced)
        tp_ms = e0t.elapsed_time(e1t) / reps
        tp_bytes = (2 * K + 1) * s * N
        two_pass = {"ms_per_step": round(tp_ms, 4), "value": K * N / (tp_ms / 1e3),
                    "algorithmic_bytes": tp_bytes, "GBps": round(tp_bytes / (tp_ms / 1e3) / 1e9, 1),
                    "frac": round(tp_bytes / (tp_ms / 1e3) / 1e9 / PEAK_HBM_GBPS, 4)}
        log(f"two-pass resolve on the same inputs: {tp_ms:.3f} ms/step ({two_pass['GBps']} GB/s)")

    # per-bucket conflict diagnostics on the step's Gram matrices: outside the
    # step (they read only the B*K*K Gram), timed on their own
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    bkmoo.conflicts(G)
    e0.record(stream)
    for _ in range(20):
        bkmoo.conflicts(G)
    e1.record(stream)
    torch.cuda.synchronize()
    extras = {"conflicts": round(e0.elapsed_time(e1) / 20, 4)}
    log(f"conflict diagnostics: {extras['conflicts'] * 1e3:.1f} us for {B} buckets")

    # the exact solvers (support enumeration) on the step's Gram matrices, and
    # at their heaviest scope: K=10 with 6,564 buckets (1 MiB fp32 buckets of
    # a 1.7B-parameter model), on seeded random positive definite Grams
    def time_solve(g, method, reps=5):
        bkmoo.solve(g, method, cagrad_c=wl.cagrad_c)
        e0.record(stream)
        for _ in range(reps):
            bkmoo.solve(g, method, cagrad_c=wl.cagrad_c)
        e1.record(stream)
        torch.cuda.synchronize()
        return round(e0.elapsed_time(e1) / reps, 4)

    if K <= 10:
        extras["solve_mgda_exact"] = time_solve(G, "mgda-exact")
        extras["solve_cagrad_exact"] = time_solve(G, "cagrad-exact")
    gen = torch.Generator(device=dev).manual_seed(1005)
    x10 = torch.randn((6564, 10, 24), generator=gen, device=dev, dtype=torch.float64)
    G10 = torch.matmul(x10, x10.transpose(1, 2).contiguous()).contiguous()
    extras["solve_mgda_exact_k10_b6564"] = time_solve(G10, "mgda-exact", reps=2)
    extras["solve_cagrad_exact_k10_b6564"] = time_solve(G10, "cagrad-exact", reps=2)
    log("exact solvers (ms): " + ", ".join(f"{k} {v:.3f}" for k, v in extras.items() if "exact" in k))

    # the sliced mode at this shape (every bucket cut into 8 slices: the
    # Gram pass over 8*B slice offsets, then the slice-order reduction) and
    # global MOO (one bucket for all N); both read K*s*N bytes
    so8 = bkmoo.slice_offsets(offs, 8)
    ws8 = torch.empty(bkmoo.workspace_size(K, N, 8 * B, wl.dtype), dtype=torch.uint8, device=dev)
    P8 = torch.empty((B, 8, K, K), dtype=torch.float64, device=dev)
    G8 = torch.empty((B, K, K), dtype=torch.float64, device=dev)
    offs1 = torch.tensor([0, N], dtype=torch.int64, device=dev)
    ws1 = torch.empty(bkmoo.workspace_size(K, N, 1, wl.dtype), dtype=torch.uint8, device=dev)
    G1 = torch.empty((1, K, K), dtype=torch.float64, device=dev)

    def sliced():
        bkmoo.gram(grads, so8, gram_out=P8.view(8 * B, K, K), workspace=ws8)
        bkmoo.gram_reduce(P8, bkmoo.SLICES_BUCKET_MAJOR, gram_out=G8)

    for name, fn in (("gram_sliced_T8", sliced),
                     ("gram_global_B1", lambda: bkmoo.gram(grads, offs1, gram_out=G1, workspace=ws1))):
        fn()
        e0.record(stream)
        for _ in range(3):
            fn()
        e1.record(stream)
        torch.cuda.synchronize()
        extras[name] = round(e0.elapsed_time(e1) / 3, 4)
    per_bucket = f", per-bucket Gram {st['gram']:.3f} ms" if "gram" in st else ""
    log(f"sliced Gram (T=8) {extras['gram_sliced_T8']:.3f} ms, global Gram (B=1) "
        f"{extras['gram_global_B1']:.3f} ms{per_bucket}")
    del ws8, P8, ws1

    # dominant kernel: the cooperative kernel (credited with the one-read
    # floor: the gradients once and the update), or the longer of the two
    # streaming passes
    if cooperative:
        kname, kbytes, kms = path_name, (K + 1) * s * N, st["resolve"]
    elif st["combine"] >= st["gram"]:
        kname, kbytes, kms = "combine", (K + 1) * s * N, st["combine"]
    else:
        kname, kbytes, kms = "gram", K * s * N, st["gram"]
    achieved = kbytes / (kms / 1e3) / 1e9
    traffic = committed_traffic(wl.name, kname)
    roof = {"bound": "hbm", "achieved": round(achieved, 1), "peak": PEAK_HBM_GBPS, "unit": "GB/s",
            "frac": round(achieved / PEAK_HBM_GBPS, 4), "traffic": traffic,
            "traffic_kind": "L2-to-fabric bytes (FETCH_SIZE + WRITE_SIZE): Infinity Cache hits included",
            "kernel": kname, "algorithmic_bytes_per_launch": kbytes, "avg_launch_ms": round(kms, 4)}
    if traffic is not None:
        # DRAM bytes lie between the bytes the kernel must move and what it
        # drew through the fabric
        roof["dram_bytes_bounds"] = [kbytes, max(traffic, kbytes)]
    if cooperative:
        # what the kernel draws from memory (one read, the second read of the
        # part it did not keep on chip, the update) over peak, beside the
        # one-read credit above
        roof["requested_bytes_per_launch"] = traffic_bytes
        roof["requested_frac"] = round(traffic_bytes / (kms / 1e3) / 1e9 / PEAK_HBM_GBPS, 4)
    result = {
        "metric": METRIC,
        "value": K * N / (ms_step / 1e3),
        "unit": "elem/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": wl.dtype,
        "data": "synthetic",
        "config": {"workload": wl.name, "K": K, "N": N, "B": B, "bucket_elems": wl.bucket_elems,
                   "method": wl.method, "max_iter": wl.max_iter, "cagrad_c": wl.cagrad_c},
        "path": path_name,
        "stages_ms": {k: round(v, 4) for k, v in st.items()},
        "extras_ms": extras,
        "resolve_requested_bytes": traffic_bytes,
        "resolve_requested_GBps": round(traffic_bytes / (ms_step / 1e3) / 1e9, 1),
        "roofline": roof,
    }
    if two_pass is not None:
        result["two_pass"] = two_pass
    if not args.no_cpu_baseline:
        log(f"oracle CPU baseline, ~{args.cpu_seconds:.0f} s")
        result["cpu_baseline"] = cpu_baseline(wl, grads, args.cpu_seconds)
    # release the device buffers and let the queued work finish before the
    # interpreter tears down
    del grads, out, ws, G, W, A
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
