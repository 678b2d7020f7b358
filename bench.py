"""Benchmark of the clustered / improved-clustered attention forward pass.

Default line: one step = one clustered forward and one improved-clustered
forward over the length-sweep workload at N = 32768 (batch 1, 8 heads, d 64,
fp32, iid N(0, 1) queries, keys and values, C = 100, 63-bit hashes, 10 Lloyd
rounds, top-32 keys), i.e. every stage of both variants on the largest
single-GPU configuration that runs both of them.  --speech gives the same line
on the speech-encoder-shaped workload (32 x 6 x 800, ragged lengths, d 32).
Inputs are seeded synthetic data already resident in HBM.

Prints one JSON line.  value = queries answered per second, counting each
valid (sequence, head, position) once per variant.  The roofline entry times
the largest kernel among the hash, centroid-attention and output stages (the
centroid GEMMs of the improved call on the default workload) with HIP events
recorded by the library around it on the call's stream, in every eighth timed
step; the K-means stage, whose time is set by its dependent rounds rather
than by a roofline, is left to "phases" unless --stage kmeans asks for it.
"phases" gives every stage's achieved rate against its bound; the
cpu_baseline entry times the fp64 oracle on the host's cores on the same
workload.
"""
from __future__ import annotations

import argparse
import ctypes
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAKS = {  # MI355X published peaks
    "hbm_GBps": 8000.0,
    "fp32_mfma_TFLOPs": 157.3,
    "bf16_mfma_TFLOPs": 2500.0,
    "int8_mfma_TOPs": 5000.0,
    "fp64_TFLOPs": 78.6,
}


class Hip:
    """Minimal HIP event API through ctypes (events on an explicit stream)."""

    def __init__(self):
        self.lib = ctypes.CDLL("libamdhip64.so")
        self.lib.hipEventCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
        self.lib.hipEventCreateWithFlags.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_uint]
        self.lib.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
        self.lib.hipEventSynchronize.argtypes = [ctypes.c_void_p]
        self.lib.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p,
                                                 ctypes.c_void_p]
        self.lib.hipEventDestroy.argtypes = [ctypes.c_void_p]

    def event(self, light=False):
        """A timing event.  light: without the system-scope fence on record
        (hipEventDisableSystemFence), so that recording it between two kernels
        does not stall the stream on a cache write-back; its timestamps are
        unaffected."""
        ev = ctypes.c_void_p()
        if light:
            assert self.lib.hipEventCreateWithFlags(ctypes.byref(ev), 0x20000000) == 0
        else:
            assert self.lib.hipEventCreate(ctypes.byref(ev)) == 0
        return ev

    def record(self, ev, stream):
        assert self.lib.hipEventRecord(ev, ctypes.c_void_p(stream)) == 0

    def elapsed_ms(self, a, b):
        """Milliseconds between two recorded events; None if they were never
        recorded (a stage that the call's path does not contain)."""
        assert self.lib.hipEventSynchronize(b) == 0
        ms = ctypes.c_float()
        if self.lib.hipEventElapsedTime(ctypes.byref(ms), a, b) != 0:
            self.lib.hipGetLastError()  # clear the error state of the failed query
            return None
        return float(ms.value)

    def destroy(self, ev):
        self.lib.hipEventDestroy(ev)


COMPUTE_UNITS = 256  # MI355X; bench_forward reads the device's own count


def fused_centroid_sums(w, compute_units=None):
    """Whether the library forms the per-workgroup centroid sums inside the
    one-launch K-means: sequences longer than 4096 (the several-workgroup
    driver, 2048 queries per workgroup) whose grid covers every compute
    unit.  The centroid stage then only adds the workgroups' parts."""
    B, H, N, _ = w.q.shape
    if N <= 4096:
        return False
    nwg = (N + 2047) // 2048
    return B * H * nwg >= (compute_units or COMPUTE_UNITS)


def stage_work(w, stage, variant_topk, compute_units=None):
    """Algorithmic work of one launch of a stage over the whole batch:
    returns (amount, unit, bound, peak) for the roofline entry.  Per
    (sequence, head) of valid length n, with C_eff = min(C, n):
      hash: read Q, write the codes (n d s + 8 n bytes);
      kmeans: L n C_eff Hamming distances, each a 64-entry int8 dot product
        on the matrix cores (2 * 64 operations);
      centroids: gather Q once, read the member list (n d s + 4 n bytes);
        when the K-means kernel gathers Q itself (fused_centroid_sums), read
        the workgroups' fp64 parts (C W d 8 bytes, W workgroups) instead;
      centroid attention (the tile kernel, or tile + merge): Q^c K^T and A^c V,
        2 C_eff n d flops each;
      output: clustered, write every row and read the assignment (n d s + 4 n);
        improved, gather Q and the T rows of K and V (C_eff k rows each), write
        every row."""
    H = w.q.shape[1]
    D = w.q.shape[3]
    lens = w.lengths.astype(np.int64)
    nsum = int(lens.sum()) * H                                   # valid queries = valid keys
    cn = int((np.minimum(lens, w.C) * lens).sum()) * H          # sum over units of C_eff n
    ceff = int(np.minimum(lens, w.C).sum()) * H                 # sum over units of C_eff
    s = 4 if w.dtype == "f32" else 2
    if stage in ("centroid_attn", "attn_tile"):
        flops = 4.0 * cn * D
        peak = PEAKS["fp32_mfma_TFLOPs"] if w.dtype == "f32" else PEAKS["bf16_mfma_TFLOPs"]
        return flops, "TFLOP/s", "mfma", peak
    if stage == "kmeans":
        ops = 2.0 * 64 * w.L * cn
        return ops, "TOP/s", "mfma", PEAKS["int8_mfma_TOPs"]
    if stage == "hash":
        byts = nsum * D * s + nsum * 8
        return byts, "GB/s", "hbm", PEAKS["hbm_GBps"]
    if stage == "output":
        if variant_topk:
            kk = np.minimum(lens, variant_topk)
            trow = int((np.minimum(lens, w.C) * kk).sum()) * H   # sum of C_eff k_eff
            byts = 2 * nsum * D * s + 2 * trow * D * s
        else:
            byts = nsum * D * s + nsum * 4
        return byts, "GB/s", "hbm", PEAKS["hbm_GBps"]
    if stage == "centroids":
        if fused_centroid_sums(w, compute_units):
            units = w.q.shape[0] * H
            nwg = (w.q.shape[2] + 2047) // 2048
            byts = units * w.C * nwg * D * 8 + ceff * D * 4 + units * w.C * 4
        else:
            byts = nsum * D * s + nsum * 4 + ceff * D * 4
        return byts, "GB/s", "hbm", PEAKS["hbm_GBps"]
    raise ValueError(stage)


def kernel_source_hash():
    """sha256 over the library's kernel sources (file names and contents)."""
    import hashlib
    d = os.path.join(ROOT, "paper_2007_04825_amd", "csrc")
    h = hashlib.sha256()
    for name in sorted(os.listdir(d)):
        if name.endswith((".hip", ".h")):
            h.update(name.encode())
            with open(os.path.join(d, name), "rb") as f:
                h.update(f.read())
    return h.hexdigest()


def measured_traffic(kernel_key, profile="speech_b32h6n800_d32_f32"):
    """HBM bytes per launch of the given kernel from the committed counter
    profile of the workload (FETCH_SIZE and WRITE_SIZE, each scaled by the same
    counter's reading for a plain copy of known size), or None when there is no
    such profile or the kernel sources changed after it was taken."""
    path = os.path.join(ROOT, "profiles", profile + "_hbm_counters.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        prof = json.load(f)
    if prof.get("source_sha256") != kernel_source_hash():
        return None
    entry = prof.get("kernels", {}).get(kernel_key)
    return None if entry is None else entry.get("hbm_bytes_per_launch")


def cpu_threads():
    """Host threads for the oracle: the CPU share of this process (its affinity
    mask, capped by OMP_NUM_THREADS when set)."""
    n = len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else (os.cpu_count() or 1)
    omp = os.environ.get("OMP_NUM_THREADS", "")
    if omp.isdigit() and int(omp) > 0:
        n = min(n, int(omp))
    return max(n, 1)


def cpu_baseline(w, min_seconds=10.0, max_passes=1000):
    """Times the fp64 oracle (both variants) on the same workload for at
    least min_seconds.  The oracle runs the (sequence, head) units in
    parallel, so it uses min(host threads, units) threads."""
    import oracle
    threads = min(cpu_threads(), w.q.shape[0] * w.q.shape[1])
    q = np.nan_to_num(w.q, nan=0.0)
    oracle.forward(q[:1], w.k[:1], w.v[:1], w.lengths[:1], w.planes, w.C, w.n_bits, w.L, w.topk,
                   num_threads=threads, exports=False)  # load / warm
    passes, t0 = 0, time.perf_counter()
    while True:
        for topk in (0, w.topk):
            oracle.forward(q, w.k, w.v, w.lengths, w.planes, w.C, w.n_bits, w.L, topk,
                           num_threads=threads, exports=False)
        passes += 1
        el = time.perf_counter() - t0
        if el >= min_seconds or passes >= max_passes:
            break
    queries = 2 * w.queries() * passes
    return {"value": queries / el, "unit": "queries/s", "cores": threads, "kind": "oracle",
            "cpu": cpu_model(),
            "sample": "%d passes of the full workload, both variants (%.1f s)" % (passes, el)}


def cpu_baseline_backward(w, fwd_exports, dout, min_seconds=10.0, max_passes=1000):
    """Times the fp64 oracle's backward pass (both variants) on the same
    workload, partitions and top-k sets, for at least min_seconds."""
    import oracle
    threads = cpu_threads()
    q = np.nan_to_num(w.q, nan=0.0)
    passes, t0 = 0, time.perf_counter()
    while True:
        for topk, fx in fwd_exports:
            oracle.backward(q, w.k, w.v, w.lengths, w.C, topk, fx["assign"], fx["topk"] if topk else None,
                            dout, num_threads=threads)
        passes += 1
        el = time.perf_counter() - t0
        if el >= min_seconds or passes >= max_passes:
            break
    queries = 2 * w.queries() * passes
    return {"value": queries / el, "unit": "queries/s", "cores": threads, "kind": "oracle",
            "sample": "%d passes of the full workload's backward, both variants (%.1f s)" % (passes, el)}


def bench_backward(args):
    """Times one backward step: the clustered and the improved backward pass
    over the speech workload, each for the forward call whose workspace it
    reads (both forwards run once before the timed region)."""
    import torch

    import gen
    import paper_2007_04825_amd as ca

    w = gen.make_config(2)
    B, H, N, D = w.q.shape
    dev = torch.device("cuda:0")
    q, k, v = (torch.from_numpy(x).to(dev) for x in (w.q, w.k, w.v))
    planes = torch.from_numpy(w.planes).to(dev)
    lengths = torch.from_numpy(w.lengths).to(dev)
    dout_np = gen.output_gradient(w)
    dout = torch.from_numpy(dout_np).to(dev)
    U = B * H
    ws, bws, grads, exports = {}, {}, {}, []
    for topk in (0, w.topk):
        ws[topk] = torch.empty(ca.workspace_bytes(B, H, N, D, 0, w.C, w.n_bits, topk), dtype=torch.uint8,
                               device=dev)
        bws[topk] = torch.empty(ca.backward_workspace_bytes(B, H, N, D, 0, w.C, topk), dtype=torch.uint8,
                                device=dev)
        grads[topk] = tuple(torch.empty_like(q) for _ in range(3))
        ex = {"assign_out": torch.zeros((U, N), dtype=torch.int32, device=dev),
              "topk_out": torch.zeros((U, w.C, max(topk, 1)), dtype=torch.int32, device=dev)}
        aux = ca.make_aux(**ex)
        if topk:
            ca.iclustered_attention(q, k, v, planes, w.C, w.n_bits, w.L, topk, lengths=lengths,
                                    workspace=ws[topk], aux=aux)
        else:
            ca.clustered_attention(q, k, v, planes, w.C, w.n_bits, w.L, lengths=lengths,
                                   workspace=ws[topk], aux=aux)
        torch.cuda.synchronize()
        exports.append((topk, {"assign": ex["assign_out"].cpu().numpy().reshape(B, H, N),
                               "topk": ex["topk_out"].cpu().numpy().reshape(B, H, w.C, max(topk, 1))}))

    def bwd(topk):
        if topk:
            ca.iclustered_attention_backward(q, k, v, dout, w.C, topk, ws[topk], lengths=lengths,
                                             bwd_workspace=bws[topk], grads=grads[topk])
        else:
            ca.clustered_attention_backward(q, k, v, dout, w.C, ws[topk], lengths=lengths,
                                            bwd_workspace=bws[topk], grads=grads[topk])

    hip = Hip()
    stream = torch.cuda.current_stream(dev).cuda_stream
    lib = ca.library()
    for _ in range(args.warmup):
        bwd(0)
        bwd(w.topk)
    torch.cuda.synchronize()
    # which variant's centroid kernel is larger
    tk = {}
    for topk in (0, w.topk):
        e0, e1 = hip.event(), hip.event()
        assert lib.ca_time_next_stage(ca.CA_KERNEL_BWD_CENTROID, e0, e1) == 0
        bwd(topk)
        tk[topk] = hip.elapsed_ms(e0, e1)
    var = max(tk, key=tk.get)
    EV_EVERY = 8
    evs = [(hip.event(light=True), hip.event(light=True)) if i % EV_EVERY == 0 else None
           for i in range(args.steps)]
    t_start, t_stop = hip.event(), hip.event()
    torch.cuda.synchronize()
    hip.record(t_start, stream)
    for i in range(args.steps):
        for topk in (0, w.topk):
            if topk == var and evs[i] is not None:
                assert lib.ca_time_next_stage(ca.CA_KERNEL_BWD_CENTROID, evs[i][0], evs[i][1]) == 0
            bwd(topk)
    hip.record(t_stop, stream)
    torch.cuda.synchronize()
    ms_per_step = hip.elapsed_ms(t_start, t_stop) / args.steps
    timed = [e for e in evs if e is not None]
    stage_ms = sum(hip.elapsed_ms(a, b) for a, b in timed) / len(timed)
    nsum = int(w.lengths.astype(np.int64).sum()) * H
    flops = 10.0 * w.C * nsum * D  # five C x n x d products per unit (S, gA, dQ^c, dK, dV)
    achieved = flops / (stage_ms * 1e-3) / 1e12
    peak = PEAKS["fp32_mfma_TFLOPs"]
    kernel_key = "bwd_centroid (%s)" % ("iclustered" if var else "clustered")
    cpu = None if args.no_cpu_baseline else cpu_baseline_backward(w, exports, dout_np)
    rec = {
        "metric": "gradient queries/sec/GPU of clustered & i-clustered attn bwd",
        "value": round(2 * w.queries() / (ms_per_step * 1e-3), 1),
        "unit": "queries/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": "speech-encoder layer: batch 32, heads 6, N 800 (lengths 400-800), "
                               "d 32, fp32, C 100, k 32; backward of clustered + i-clustered",
                   "global_batch": B, "seq_len": N, "parallelism": "none"},
        "roofline": {"bound": "mfma", "achieved": round(achieved, 3), "peak": peak, "unit": "TFLOP/s",
                     "frac": round(achieved / peak, 5), "traffic": measured_traffic(kernel_key),
                     "kernel": kernel_key, "avg_launch_us": round(stage_ms * 1e3, 3)},
        "cpu_baseline": cpu,
    }
    print(json.dumps(rec))


def _timed(hip, stream, fn, reps):
    """Median of reps HIP-event timings of fn (ms) after three untimed calls."""
    import torch
    for _ in range(3):
        fn()
    torch.cuda.synchronize()
    ts = []
    for _ in range(reps):
        e0, e1 = hip.event(), hip.event()
        hip.record(e0, stream)
        fn()
        hip.record(e1, stream)
        ts.append(hip.elapsed_ms(e0, e1))
        hip.destroy(e0)
        hip.destroy(e1)
    return float(np.median(ts))


def _length_point(w, reps, hip, stream, exact_batch=None):
    """Times one workload at one length: each variant's forward and forward +
    backward, and (exact_batch > 0) torch's fp32 scaled_dot_product_attention
    with its autograd backward on the first exact_batch sequences.  Returns
    {name: (ms, peak bytes beyond the resident inputs, sequences)}; the peak
    covers the workspaces, outputs and gradients that each path allocates
    through torch."""
    import torch

    import gen
    import paper_2007_04825_amd as ca

    dev = torch.device("cuda:0")
    B, H, N, D = w.q.shape
    dt = ca.CA_F32 if w.dtype == "f32" else ca.CA_BF16
    tdt = torch.float32 if w.dtype == "f32" else torch.bfloat16
    q, k, v = (torch.from_numpy(x).to(dev).to(tdt) for x in (w.q, w.k, w.v))
    planes = torch.from_numpy(w.planes).to(dev)
    dout = torch.from_numpy(gen.output_gradient(w)).to(dev).to(tdt)
    res = {}

    def peak_of(run):
        torch.cuda.synchronize()
        base = torch.cuda.memory_allocated()
        torch.cuda.reset_peak_memory_stats()
        run()
        torch.cuda.synchronize()
        return torch.cuda.max_memory_allocated() - base

    for name, topk in (("clustered", 0), ("iclustered", w.topk)):
        state = {}

        def alloc():
            state["ws"] = torch.empty(ca.workspace_bytes(B, H, N, D, dt, w.C, w.n_bits, topk),
                                      dtype=torch.uint8, device=dev)
            state["bws"] = torch.empty(ca.backward_workspace_bytes(B, H, N, D, dt, w.C, topk),
                                       dtype=torch.uint8, device=dev)
            state["out"] = torch.empty_like(q)
            state["grads"] = tuple(torch.empty(q.shape, dtype=torch.float32, device=dev) for _ in range(3))

        def fwd():
            if topk:
                ca.iclustered_attention(q, k, v, planes, w.C, w.n_bits, w.L, topk, out=state["out"],
                                        workspace=state["ws"])
            else:
                ca.clustered_attention(q, k, v, planes, w.C, w.n_bits, w.L, out=state["out"],
                                       workspace=state["ws"])

        def fwd_bwd():
            fwd()
            if topk:
                ca.iclustered_attention_backward(q, k, v, dout, w.C, topk, state["ws"],
                                                 bwd_workspace=state["bws"], grads=state["grads"])
            else:
                ca.clustered_attention_backward(q, k, v, dout, w.C, state["ws"],
                                                bwd_workspace=state["bws"], grads=state["grads"])

        mem = peak_of(lambda: (alloc(), fwd_bwd()))
        res[name + "_fwd"] = (_timed(hip, stream, fwd, reps), None, B)
        res[name + "_fwd_bwd"] = (_timed(hip, stream, fwd_bwd, reps), mem, B)
        state.clear()
    if exact_batch:
        be = min(B, exact_batch)
        tq, tk, tv = (x[:be].float().clone().requires_grad_(True) for x in (q, k, v))
        g32 = dout[:be].float().contiguous()

        def exact_fwd():
            with torch.no_grad():
                torch.nn.functional.scaled_dot_product_attention(tq, tk, tv)

        def exact_fwd_bwd():
            o = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv)
            o.backward(g32)

        res["exact_fwd"] = (_timed(hip, stream, exact_fwd, reps), None, be)
        mem = peak_of(exact_fwd_bwd)
        for x in (tq, tk, tv):
            x.grad = None
        res["exact_fwd_bwd"] = (_timed(hip, stream, exact_fwd_bwd, reps), mem, be)
        del tq, tk, tv, g32
    del q, k, v, planes, dout
    torch.cuda.empty_cache()
    return res


def bench_sweep(args):
    """Length sweep: batch 1, 8 heads x 64, N = 2^10 .. 2^15, fp32 and bf16
    storage (iid N(0, 1) inputs, C 100, B 63, L 10, k 32); each variant's
    forward and forward + backward timed with HIP events (median of repetitions
    after warm-up) next to exact softmax attention (torch's fp32
    scaled_dot_product_attention, its backward through autograd).  One JSON
    line per (N, dtype) with times per (query, head)."""
    import torch

    import gen

    dev = torch.device("cuda:0")
    hip = Hip()
    stream = torch.cuda.current_stream(dev).cuda_stream
    for dtype in ("f32", "bf16"):
        for logn in range(10, 16):
            N = 1 << logn
            w = gen.config_sweep(N, dtype=dtype)
            B, H, _, D = w.q.shape
            res = _length_point(w, 20 if N <= 8192 else 8, hip, stream,
                                exact_batch=B if dtype == "f32" else None)
            rec = {"N": N, "heads": H, "d": D, "dtype": dtype, "unit": "us per (query, head)"}
            for key, (ms, _, nb) in res.items():
                rec[key] = round(ms * 1e3 / (nb * N * H), 6)
            print(json.dumps(rec), flush=True)


def bench_fig4(args):
    """The paper's time and memory benchmark protocol: one attention layer of
    6 heads x 64, N = 2^9 .. 2^15, as many sequences per call as the path is
    given (a budget of 2^17 tokens, so batch = 2^17 / N), C 100, B 63, L 10,
    k 32, fp32, iid N(0, 1) inputs.  Reports GPU time and the peak memory
    beyond the resident inputs per sequence element, forward and forward +
    backward, for both variants and exact attention.  Exact attention takes at
    most 2^32 / (6 N^2) sequences per call (at least one), which keeps one
    N x N fp32 tensor per call under 17 GB whichever backend torch picks.  The
    projections and the feed-forward layer of the paper's one-layer model lie
    outside the path and are not timed."""
    import torch

    import gen

    dev = torch.device("cuda:0")
    hip = Hip()
    stream = torch.cuda.current_stream(dev).cuda_stream
    budget = 1 << 17
    for logn in range(9, 16):
        N = 1 << logn
        B = max(1, budget // N)
        w = gen.config_sweep(N, dtype="f32", B=B, H=6, d=64)
        be = max(1, min(B, (1 << 32) // (6 * N * N)))
        res = _length_point(w, 10 if N <= 4096 else 5, hip, stream, exact_batch=be)
        rec = {"N": N, "batch": B, "exact_batch": be, "heads": 6, "d": 64, "dtype": "f32",
               "unit": "us per element; bytes per element"}
        for key, (ms, mem, nb) in res.items():
            rec[key + "_us"] = round(ms * 1e3 / (nb * N), 6)
            if mem is not None:
                rec[key + "_bytes"] = round(mem / (nb * N), 1)
        print(json.dumps(rec), flush=True)


def bench_long(args):
    """Long-context stress: batch 1, 8 heads x 64, N = 65536, bf16 storage,
    C 200, B 63, L 15, k 64, improved clustered attention only.  One JSON line:
    the forward's time (median of HIP-event timings), queries per second, and
    each stage's time from separate calls."""
    import torch

    import gen
    import paper_2007_04825_amd as ca

    dev = torch.device("cuda:0")
    global COMPUTE_UNITS
    COMPUTE_UNITS = torch.cuda.get_device_properties(dev).multi_processor_count
    hip = Hip()
    stream = torch.cuda.current_stream(dev).cuda_stream
    w = gen.config_long()
    B, H, N, D = w.q.shape
    q, k, v = (torch.from_numpy(x).to(dev).to(torch.bfloat16) for x in (w.q, w.k, w.v))
    planes = torch.from_numpy(w.planes).to(dev)
    ws = torch.empty(ca.workspace_bytes(B, H, N, D, ca.CA_BF16, w.C, w.n_bits, w.topk),
                     dtype=torch.uint8, device=dev)
    out = torch.empty_like(q)

    def fwd():
        ca.iclustered_attention(q, k, v, planes, w.C, w.n_bits, w.L, w.topk, out=out, workspace=ws)

    ms = _timed(hip, stream, fwd, max(3, args.steps // 20))
    stages = {}
    lib = ca.library()
    for name, sid in dict(ca.STAGES, attn_tile=ca.CA_KERNEL_ATTN_TILE).items():
        ts = []
        for _ in range(3):
            e0, e1 = hip.event(), hip.event()
            assert lib.ca_time_next_stage(sid, e0, e1) == 0
            fwd()
            t = hip.elapsed_ms(e0, e1)
            hip.destroy(e0)
            hip.destroy(e1)
            if t is None:
                break
            ts.append(t)
        if ts:
            stages[name] = round(float(np.median(ts)) * 1e3, 1)
    print(json.dumps({"metric": "queries/sec/GPU of i-clustered attn fwd (long context)",
                      "value": round(B * N / (ms * 1e-3), 1), "unit": "queries/s",
                      "ms_per_call": round(ms, 4), "dtype": "bf16", "data": "synthetic",
                      "config": {"workload": "long-context stress: batch 1, heads 8, N 65536, d 64, bf16, "
                                             "C 200, B 63, L 15, k 64; i-clustered"},
                      "stages_us": stages,
                      "phases": {name: phase_entry(w, name, w.topk, us, LONG_PROFILE)
                                 for name, us in stages.items() if name != "centroid_attn"}}),
          flush=True)


def bench_oracle_top(args):
    """Oracle-top attention (each query keeps its k = 32 keys of highest logit)
    on the speech-encoder workload: one JSON line with the throughput, the
    roofline entry of its tile kernel (the n x n logits on the fp32 matrix
    cores, 2 n^2 d flops per (sequence, head); the top-k rows add 2 n k d) and
    the fp64 oracle timed on the host."""
    import torch

    import gen
    import oracle
    import paper_2007_04825_amd as ca

    w = gen.make_config(2)
    B, H, N, D = w.q.shape
    dev = torch.device("cuda:0")
    hip = Hip()
    stream = torch.cuda.current_stream(dev).cuda_stream
    q, k, v = (torch.from_numpy(x).to(dev) for x in (w.q, w.k, w.v))
    lengths = torch.from_numpy(w.lengths).to(dev)
    ws = torch.empty(ca.oracle_top_workspace_bytes(B, H, N, D, ca.CA_F32, w.topk), dtype=torch.uint8,
                     device=dev)
    out = torch.empty_like(q)

    def step():
        ca.oracle_top_attention(q, k, v, w.topk, lengths=lengths, out=out, workspace=ws)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    e0, e1 = hip.event(), hip.event()
    hip.record(e0, stream)
    for _ in range(args.steps):
        step()
    hip.record(e1, stream)
    ms = hip.elapsed_ms(e0, e1) / args.steps
    # the tile kernel alone, from the library's event hook
    lib = ca.library()
    kts = []
    for _ in range(20):
        a0, a1 = hip.event(), hip.event()
        assert lib.ca_time_next_stage(ca.CA_KERNEL_CENTROID_ATTN, a0, a1) == 0
        step()
        kts.append(hip.elapsed_ms(a0, a1))
        hip.destroy(a0)
        hip.destroy(a1)
    kus = float(np.mean(kts)) * 1e3
    lens = w.lengths.astype(np.float64)
    flops = float(H * (2.0 * (lens ** 2).sum() * D + 2.0 * lens.sum() * w.topk * D))
    achieved = flops / (kus * 1e-6) / 1e12
    nq = int(w.lengths.sum()) * H
    rec = {"metric": "queries/sec/GPU of oracle-top attn fwd", "value": round(nq / (ms * 1e-3), 1),
           "unit": "queries/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
           "ms_per_step": round(ms, 5), "higher_is_better": True, "dtype": "f32",
           "data": "synthetic",
           "config": {"workload": "speech-encoder layer: batch 32, heads 6, N 800 (lengths 400-800), "
                                  "d 32, fp32, k 32; oracle-top"},
           "roofline": {"bound": "mfma", "achieved": round(achieved, 3),
                        "peak": PEAKS["fp32_mfma_TFLOPs"], "unit": "TFLOP/s",
                        "frac": round(achieved / PEAKS["fp32_mfma_TFLOPs"], 5), "traffic": None,
                        "kernel": "attn_tile_kernel (oracle-top)", "avg_launch_us": round(kus, 3)}}
    if not args.no_cpu_baseline:
        threads = cpu_threads()
        passes, t0 = 0, time.perf_counter()
        while True:
            oracle.oracle_top(w.q, w.k, w.v, w.lengths, w.topk, num_threads=threads)
            passes += 1
            el = time.perf_counter() - t0
            if el >= 10.0:
                break
        rec["cpu_baseline"] = {"value": round(nq * passes / el, 1), "unit": "queries/s",
                               "cores": threads, "kind": "oracle",
                               "sample": "%d passes of the full workload (%.1f s)" % (passes, el)}
    print(json.dumps(rec), flush=True)


def copy_calibration(nbytes):
    """A plain device-to-device copy of known size, for scaling HBM counters."""
    import torch
    a = torch.ones(nbytes // 4, dtype=torch.float32, device="cuda")
    b = torch.empty_like(a)
    for _ in range(5):
        b.copy_(a)
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration_bytes": nbytes}))


def cpu_model():
    """The host CPU's model name (from /proc/cpuinfo), or the platform string."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    import platform
    return platform.processor() or platform.machine()


def phase_entry(w, stage, variant_topk, us, profile=None):
    """Achieved rate of one stage launch (the whole batch) against its bound,
    and the stage's HBM bytes per launch from the workload's committed counter
    profile (null without one, or once the kernels have changed)."""
    amount, unit, bound, peak = stage_work(w, stage, variant_topk)
    if us is None or us <= 0:
        return None
    achieved = amount / (us * 1e-6) / (1e9 if unit == "GB/s" else 1e12)
    key = "%s (%s)" % (stage, "iclustered" if variant_topk else "clustered")
    return {"us": round(us, 2), "achieved": round(achieved, 3), "unit": unit, "bound": bound,
            "peak": peak, "frac": round(achieved / peak, 5),
            "traffic": measured_traffic(key, profile) if profile else None}


HEADLINE = {
    "workload": "length-sweep point: batch 1, heads 8, N 32768, d 64, fp32, iid N(0,1) Q/K/V, "
                "C 100, B 63, L 10, k 32; clustered + i-clustered",
    "profile": "sweep_b1h8n32768_d64_f32",
}
LONG_PROFILE = "long_b1h8n65536_d64_bf16"
SPEECH = {
    "workload": "speech-encoder layer: batch 32, heads 6, N 800 (lengths 400-800), d 32, fp32, "
                "C 100, B 63, L 10, k 32; clustered + i-clustered",
    "profile": "speech_b32h6n800_d32_f32",
}


def bench_forward(args, w, desc):
    """One step = one clustered and one improved-clustered forward call over
    the whole batch of workload w (inputs resident in HBM).  Prints the
    headline JSON line: value = valid queries answered per second (each
    variant counted), over exactly args.steps back-to-back steps between two
    events; the roofline entry of the largest hash, tile or output kernel
    (the K-means with --stage kmeans), timed with event pairs
    that the library records around it on the call's stream in every eighth
    timed step; every stage's achieved rate; the per-step median of separately
    timed steps; and the fp64 oracle on the host's cores."""
    import torch

    import paper_2007_04825_amd as ca

    B, H, N, D = w.q.shape
    dt = ca.CA_F32 if w.dtype == "f32" else ca.CA_BF16
    tdt = torch.float32 if w.dtype == "f32" else torch.bfloat16
    dev = torch.device("cuda:0")
    global COMPUTE_UNITS
    COMPUTE_UNITS = torch.cuda.get_device_properties(dev).multi_processor_count
    q, k, v = (torch.from_numpy(np.nan_to_num(x, nan=0.0)).to(dev).to(tdt) for x in (w.q, w.k, w.v))
    planes = torch.from_numpy(w.planes).to(dev)
    lengths = torch.from_numpy(w.lengths).to(dev)
    ws = torch.empty(max(ca.workspace_bytes(B, H, N, D, dt, w.C, w.n_bits, w.topk),
                         ca.workspace_bytes(B, H, N, D, dt, w.C, w.n_bits, 0)),
                     dtype=torch.uint8, device=dev)
    out_c = torch.empty_like(q)
    out_i = torch.empty_like(q)
    stream = torch.cuda.current_stream(dev).cuda_stream
    hip = Hip()
    lib = ca.library()

    def call(topk):
        if topk:
            ca.iclustered_attention(q, k, v, planes, w.C, w.n_bits, w.L, topk, lengths=lengths,
                                    out=out_i, workspace=ws)
        else:
            ca.clustered_attention(q, k, v, planes, w.C, w.n_bits, w.L, lengths=lengths,
                                   out=out_c, workspace=ws)

    def step():
        call(0)
        call(w.topk)

    # per-stage times (one event pair per stage and variant, median of 5 calls)
    stages = dict(ca.STAGES)
    stages["attn_tile"] = ca.CA_KERNEL_ATTN_TILE

    def stage_times(reps=5):
        tot = {}
        for name, sid in stages.items():
            for topk in (0, w.topk):
                ts = []
                for _ in range(reps):
                    e0, e1 = hip.event(), hip.event()
                    assert lib.ca_time_next_stage(sid, e0, e1) == 0
                    call(topk)
                    ms = hip.elapsed_ms(e0, e1)
                    hip.destroy(e0)
                    hip.destroy(e1)
                    if ms is None:
                        break
                    ts.append(ms)
                if ts:
                    tot[(name, topk)] = float(np.median(ts))
        return tot

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    st = stage_times()
    # the roofline kernel: the largest of the single-kernel hash, tile and
    # output stages (the centroid stage may hold two kernels and the
    # centroid-attention stage a tile kernel and a merge; the K-means, bound
    # by its dependent rounds, only when asked for)
    single = [key for key in st if key[0] in ("hash", "attn_tile", "output")
              or (key[0] == "kmeans" and args.stage == "kmeans")]
    if args.stage == "auto":
        name, var_topk = max(single, key=st.get)
    else:
        name = args.stage
        var_topk = w.topk if st.get((name, w.topk), 0) >= st.get((name, 0), 0) else 0

    # timed region: exactly args.steps steps between two events; the dominant
    # kernel of the chosen variant is timed with its own event pair in every
    # EV_EVERY-th step (an event record between two kernels costs the stream a
    # few microseconds, which would otherwise be added to every step)
    sid = stages[name]
    EV_EVERY = 8
    evs = [(hip.event(light=True), hip.event(light=True)) if i % EV_EVERY == 0 else None
           for i in range(args.steps)]
    t_start, t_stop = hip.event(), hip.event()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    hip.record(t_start, stream)
    for i in range(args.steps):
        if var_topk == 0 and evs[i] is not None:
            assert lib.ca_time_next_stage(sid, evs[i][0], evs[i][1]) == 0
        call(0)
        if var_topk and evs[i] is not None:
            assert lib.ca_time_next_stage(sid, evs[i][0], evs[i][1]) == 0
        call(w.topk)
    hip.record(t_stop, stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    total_ms = hip.elapsed_ms(t_start, t_stop)
    timed = [e for e in evs if e is not None]
    stage_ms = sum(hip.elapsed_ms(a, b) for a, b in timed) / len(timed)
    ms_per_step = total_ms / args.steps
    queries_per_step = 2 * w.queries()
    value = queries_per_step / (ms_per_step * 1e-3)
    # per-step and per-call medians from separately timed steps
    med_step = _timed(hip, stream, step, 21)
    med_c = _timed(hip, stream, lambda: call(0), 21)
    med_i = _timed(hip, stream, lambda: call(w.topk), 21)

    amount, unit, bound, peak = stage_work(w, name, var_topk)
    achieved = amount / (stage_ms * 1e-3) / (1e12 if unit != "GB/s" else 1e9)
    kernel_key = "%s (%s)" % (name, "iclustered" if var_topk else "clustered")
    roof = {"bound": bound, "achieved": round(achieved, 3), "peak": peak, "unit": unit,
            "frac": round(achieved / peak, 5),
            "traffic": measured_traffic(kernel_key, desc["profile"]),
            "kernel": kernel_key, "avg_launch_us": round(stage_ms * 1e3, 3)}
    phases = {}
    for (n_, t_), ms in sorted(st.items()):
        if n_ == "centroid_attn":
            continue  # the tile kernel is reported alone; the merge is the difference
        e = phase_entry(w, n_, t_, ms * 1e3, desc["profile"])
        if e is not None:
            phases["%s_%s" % (n_, "ic" if t_ else "c")] = e
    for t_ in (0, w.topk):
        if ("centroid_attn", t_) in st and ("attn_tile", t_) in st:
            phases["attn_merge_%s" % ("ic" if t_ else "c")] = {
                "us": round((st[("centroid_attn", t_)] - st[("attn_tile", t_)]) * 1e3, 2)}
    cpu = None if args.no_cpu_baseline else cpu_baseline(w)
    rec = {
        "metric": "queries/sec/GPU of clustered & i-clustered attn fwd",
        "value": round(value, 1),
        "unit": "queries/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "median_ms_per_step": round(med_step, 5),
        "wall_ms_per_step": round(wall / args.steps * 1e3, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic",
        "config": {"workload": desc["workload"], "global_batch": B, "seq_len": N,
                   "parallelism": "none"},
        "per_call_median_ms": {"clustered": round(med_c, 5), "iclustered": round(med_i, 5)},
        "phases": phases,
        "roofline": roof,
        "cpu_baseline": cpu,
    }
    print(json.dumps(rec))


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--stage", default="auto",
                    choices=["auto", "hash", "kmeans", "centroids", "centroid_attn", "attn_tile",
                             "output"])
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="BYTES")
    ap.add_argument("--speech", action="store_true",
                    help="the headline line on the speech-encoder workload (32 x 6 x 800, d 32)")
    ap.add_argument("--backward", action="store_true",
                    help="time the backward pass instead (its own JSON line)")
    ap.add_argument("--sweep", action="store_true",
                    help="length sweep against exact attention (one JSON line per length)")
    ap.add_argument("--oracle-top", action="store_true",
                    help="time oracle-top attention on the speech workload (its own JSON line)")
    ap.add_argument("--long", action="store_true",
                    help="time the N = 65536 long-context forward (its own JSON line)")
    ap.add_argument("--fig4", action="store_true",
                    help="time and memory per sequence element in the paper's benchmark protocol")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU: the forward pass of each (sequence, head) is "
              "independent and the library has no multi-GPU path (--gpus %d refused)" % args.gpus,
              file=sys.stderr)
        sys.exit(2)
    if args.copy_calibration:
        copy_calibration(args.copy_calibration)
        return
    if args.backward:
        bench_backward(args)
        return
    if args.sweep:
        bench_sweep(args)
        return
    if args.fig4:
        bench_fig4(args)
        return
    if args.long:
        bench_long(args)
        return
    if args.oracle_top:
        bench_oracle_top(args)
        return

    import gen

    if args.speech:
        bench_forward(args, gen.make_config(2), SPEECH)
    else:
        bench_forward(args, gen.make_config(3, N=32768, dtype="f32"), HEADLINE)


if __name__ == "__main__":
    main()
