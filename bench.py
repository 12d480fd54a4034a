"""Throughput benchmark of the Gram-Space hot path on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload stress]

Default workload (the headline line): the stress configuration.  One bipolar
codebook of M = 2048 entries of dimension D = 16384, 205 of them duplicates of
other entries (rank 1843), is compressed once before timing (its time is
reported).  The batch holds 262144 queries x = p C + N(0, 0.1) noise with
p ~ Dirichlet(1/2), stored as bf16 (P and X), with bf16 basis and coordinates
and fp32 accumulation.  One step is the whole matrix-space pipeline over the
batch: project (t = Q x, with ||x||^2), prob2vec (t = p R), cosine similarity
with argmax and attention weights softmax(16 s) from one score product
(gs_similarity_attention), and reconstruct (x = t Q), four library calls; `value` is queries per second over the K timed
steps (synchronised wall clock), and HIP events around every call on the
launch stream give each kernel's mean duration, the dominant one going into
the matrix-core roofline entry.  The fused soft-selection step of the vsa
workload (four attribute codebooks, both of its forms) is reported under
"extra", and the oracle's rate on a seeded sample of the same batch under
"cpu_baseline".

Inputs stay resident in HBM: they are generated on the device before the
timed region, and every step reads and writes the same resident buffers
(several GB each, far beyond the 256 MiB Infinity Cache).

Other workloads (--workload): vsa makes the fused soft selection the headline
(K launches captured in one HIP graph and replayed once, cycling through
copies of the batch larger than the Infinity Cache); large and binary time one
step of the separate calls of those configurations; dimsweep measures the
similarity lookup against the vector dimension, dense and Gram-Space; bind
times the binding operators on restored vectors.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
METRIC = "coord-space similarity+prob2vec queries/s and HBM GB/s vs peak; MFMA util"
wl = None


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--workload", default="stress",
                    choices=["stress", "vsa", "large", "binary", "dimsweep", "bind", "memory"],
                    help="stress (default, the headline): the whole matrix-space pipeline of the stress "
                         "configuration in bf16; vsa: the fused soft selection of four attribute codebooks; "
                         "large / binary: the separate calls of those configurations (fp32); dimsweep: "
                         "similarity latency against the vector dimension, dense vs Gram-Space; bind: binding of "
                         "restored vectors (circular convolution / correlation, xor, product); memory: peak device "
                         "memory of each workload's operators, dense against Gram-Space")
    ap.add_argument("--steps", type=int, default=None, help="timed steps (default 20; vsa: 200)")
    ap.add_argument("--warmup", type=int, default=None, help="untimed warm-up steps (default 3; vsa: 20)")
    ap.add_argument("--sets", type=int, default=0, help="vsa: batch copies to cycle through (0: >= 1 GiB)")
    ap.add_argument("--beta", type=float, default=16.0)
    ap.add_argument("--no-cpu", action="store_true", help="skip the oracle CPU baseline")
    ap.add_argument("--cpu-seconds", type=float, default=15.0, help="vsa: seconds of oracle work to time")
    ap.add_argument("--cpu-rows", type=int, default=8192,
                    help="stress / large / binary: rows of the seeded sample the oracle processes")
    ap.add_argument("--no-vsa", action="store_true", help="stress: skip the fused vsa step reported under extra")
    ap.add_argument("--no-unfused", action="store_true", help="vsa: skip timing the 12-call path")
    ap.add_argument("--copy-probe-mib", type=int, default=0,
                    help="only run a plain device copy of this size (counter calibration)")
    ap.add_argument("--pmc-summary", nargs=4, metavar=("FETCH_CSV", "WRITE_CSV", "COPY_FETCH_CSV", "COPY_WRITE_CSV"),
                    help="turn rocprofv3 FETCH_SIZE / WRITE_SIZE counter CSVs (kernel run, copy calibration) "
                         "into profiles/traffic_<call>_<workload>.json and exit")
    ap.add_argument("--streams", type=int, default=1,
                    help="vsa: also time the fused steps spread round robin over this many streams in one "
                         "graph (independent batches in flight together, as a server would run them); reported "
                         "under extra.concurrent, not as the headline")
    ap.add_argument("--pmc-kernel", default="soft_gram_kernel",
                    help="--pmc-summary: substring of the kernel name to summarise")
    ap.add_argument("--pmc-call", default="soft_gram_kernel",
                    help="--pmc-summary: name of the call in the output file name")
    ap.add_argument("--pmc-workload", default="vsa")
    ap.add_argument("--pmc-copy-mib", type=int, default=512)
    args = ap.parse_args()
    heavy = args.workload in ("stress", "large", "binary")
    if args.steps is None:
        args.steps = 20 if heavy else 200
    if args.warmup is None:
        args.warmup = 3 if heavy else 20
    return args


def kernel_source_hash(files=None) -> str:
    """Hash of the library sources (all of csrc/, or the listed file names)."""
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2608_01528_amd", "csrc")
    names = sorted(files) if files else sorted(f for f in os.listdir(csrc) if f.endswith((".hip", ".h")))
    for f in names:
        h.update(open(os.path.join(csrc, f), "rb").read())
    return h.hexdigest()[:16]


def traffic_sources(kernel: str):
    """Source files that build a profiled kernel and its launch path (a counter
    record stays valid while these are unchanged)."""
    if "gemm256" in kernel or "scores256" in kernel:
        return ["gs_abi.hip", "gs_gemm.hip", "gs_gemm256.hip", "gs_internal.h"]
    if "soft_" in kernel:
        return ["gs_abi.hip", "gs_internal.h", "gs_small.hip"]
    if "circular_kernel" in kernel:
        return ["gs_abi.hip", "gs_bind.hip", "gs_internal.h"]
    return None


def load_traffic(call: str, workload: str):
    """HBM bytes per launch from the committed counter summary, if it was taken
    on the current sources of its kernel (else None)."""
    path = os.path.join(ROOT, "profiles", "traffic_%s_%s.json" % (call, workload))
    if not os.path.exists(path):
        return None
    try:
        d = json.load(open(path))
    except ValueError:
        return None
    if d.get("source_hash") != kernel_source_hash(d.get("sources")):
        return None
    return d.get("hbm_bytes_per_launch")


def cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


class VsaWorkload:
    """Compressed attribute codebooks and `nsets` copies of the batch."""

    def __init__(self, w, nsets, torch, gsm):
        dev = torch.device("cuda:0")
        self.w = w
        self.books = []
        self.compress_ms = []
        for i, M in enumerate(w.Ms):
            C = torch.from_numpy(wl.codebook(w, i)).to(dev)
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            Q, R, r, kept, cnorm = gsm.gs_compress(C, q_dtype=torch.float32, r_dtype=torch.float32)
            torch.cuda.synchronize()
            self.compress_ms.append((time.perf_counter() - t0) * 1e3)
            R = R.contiguous()
            P0 = torch.from_numpy(wl.probabilities(w, i)).to(dev)
            B = P0.shape[0]
            sets = []
            for s in range(nsets):
                sets.append({
                    "P": P0 if s == 0 else P0.clone(),
                    "T": torch.empty((B, r), dtype=torch.float32, device=dev),
                    "S": torch.empty((B, M), dtype=torch.float32, device=dev),
                    "argmax": torch.empty(B, dtype=torch.int32, device=dev),
                    "A": torch.empty((B, M), dtype=torch.float32, device=dev),
                })
            self.books.append({"M": M, "r": r, "R": R, "cnorm": cnorm, "sets": sets, "B": B})
        self.queries = sum(b["B"] for b in self.books)

    def fused_bytes(self):
        """Algorithmic bytes of one fused launch: read P, R, norms; write S,
        argmax, A (no coordinates are written: the Gram form never forms
        them, the coordinate form keeps them in registers)."""
        tot = 0
        for b in self.books:
            B, M, r = b["B"], b["M"], b["r"]
            tot += B * (4 * M + 4 * M + 4 + 4 * M) + 4 * M * r + 4 * M
        return tot

    def unfused_bytes(self):
        """Algorithmic bytes of the 12 separate calls (T written, then read twice)."""
        tot = 0
        for b in self.books:
            B, M, r = b["B"], b["M"], b["r"]
            cb = 4 * M * r + 4 * M
            tot += (4 * B * M + 4 * B * r + cb) + (4 * B * r + 4 * B * M + 4 * B + cb) + (4 * B * r + 4 * B * M + cb)
        return tot


def cpu_baseline_vsa(w, beta, seconds):
    """Oracle (dense fp64 in D-space) on the same workload, bounded in time:
    the row count grows until one pass over all codebooks takes a fair share
    of `seconds` (at most the whole batch), then passes repeat until about
    `seconds` of CPU work have been timed."""
    import oracle
    cores = oracle.threads()
    books = [wl.codebook(w, i) for i in range(len(w.Ms))]

    probs = {}

    def one_pass(rows):
        if rows not in probs:     # inputs are generated outside the timed region
            probs.clear()
            probs[rows] = [wl.probabilities(w, i, B=rows) for i in range(len(w.Ms))]
        t0 = time.perf_counter()
        for i in range(len(w.Ms)):
            V = oracle.prob2vec(probs[rows][i], books[i])
            S = oracle.similarity(V, books[i], oracle.COSINE)
            oracle.argmax(S)
            oracle.softmax(S, beta)
        return time.perf_counter() - t0

    rows = 256
    while True:
        dt = one_pass(rows)
        if dt >= 0.2 * seconds or rows >= w.B:
            break
        rows = min(w.B, int(rows * max(2.0, 0.25 * seconds / max(dt, 1e-3))))
    total, passes = dt, 1
    while total < seconds:
        total += one_pass(rows)
        passes += 1
    q = rows * len(w.Ms) * passes
    return {"value": q / total, "unit": "queries/s", "cores": cores, "kind": "oracle",
            "sample": "%d pass(es) over %d rows of each of the %d codebooks (%d queries): dense fp64 prob2vec, "
                      "cosine similarity, argmax and softmax in D = %d; %.1f s" % (passes, rows, len(w.Ms), q, w.D,
                                                                                    total)}


def timed_graph(torch, steps, launch_step, stream, nstreams=1):
    """Capture `steps` steps into one HIP graph and replay it once, bracketed
    by device synchronisation (wall clock) and by HIP events recorded on the
    replay stream (GPU time).  Returns (wall seconds, GPU ms per step).  With
    nstreams > 1 the steps go round robin to that many streams forked from
    and joined back into the capture stream (independent steps overlap)."""
    g = torch.cuda.CUDAGraph()
    if nstreams == 1:
        with torch.cuda.graph(g):
            for k in range(steps):
                launch_step(k)
    else:
        main = torch.cuda.Stream()
        aux = [torch.cuda.Stream() for _ in range(nstreams - 1)]
        with torch.cuda.graph(g, stream=main):
            fork = torch.cuda.Event()
            fork.record(main)
            for s_ in aux:
                s_.wait_event(fork)
            streams = [main] + aux
            for k in range(steps):
                with torch.cuda.stream(streams[k % nstreams]):
                    launch_step(k)
            for s_ in aux:
                join = torch.cuda.Event()
                join.record(s_)
                main.wait_event(join)
    g.replay()                      # warm replay (uploads the graph)
    torch.cuda.synchronize()
    a = torch.cuda.Event(enable_timing=True)
    b = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    a.record(stream)
    g.replay()
    b.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    return wall, a.elapsed_time(b) / steps


def _counter_kib(path, name_part, counter):
    """Mean per-dispatch value (KiB) of a counter for the longest dispatches of
    kernels whose name holds name_part (those lasting at least half as long as
    the longest one, so that one call is picked where two calls share a kernel
    instance), from a rocprofv3 counter_collection CSV."""
    import csv
    rows = [r for r in csv.DictReader(open(path))
            if name_part in r["Kernel_Name"] and r["Counter_Name"] == counter]
    if not rows:
        raise SystemExit("no %s records for kernels matching %r in %s" % (counter, name_part, path))
    dur = [int(r["End_Timestamp"]) - int(r["Start_Timestamp"]) for r in rows]
    keep = [float(r["Counter_Value"]) for r, d in zip(rows, dur) if d >= 0.5 * max(dur)]
    return float(np.mean(keep)), len(keep)


def pmc_summary(args):
    """HBM bytes per launch of the kernel: counter KiB x 1024, scaled by the
    ratio of true to counted bytes of a plain copy of known size."""
    fetch_csv, write_csv, cf_csv, cw_csv = args.pmc_summary
    copy_bytes = args.pmc_copy_mib * (1 << 20)
    f_kib, nf = _counter_kib(fetch_csv, args.pmc_kernel, "FETCH_SIZE")
    w_kib, nw = _counter_kib(write_csv, args.pmc_kernel, "WRITE_SIZE")
    cf_kib, _ = _counter_kib(cf_csv, "copy", "FETCH_SIZE")
    cw_kib, _ = _counter_kib(cw_csv, "copy", "WRITE_SIZE")
    f_scale = copy_bytes / (cf_kib * 1024.0)
    w_scale = copy_bytes / (cw_kib * 1024.0)
    read = f_kib * 1024.0 * f_scale
    write = w_kib * 1024.0 * w_scale
    srcs = traffic_sources(args.pmc_kernel)
    out = {"kernel": args.pmc_kernel, "call": args.pmc_call, "workload": args.pmc_workload,
           "sources": srcs, "source_hash": kernel_source_hash(srcs),
           "hbm_bytes_per_launch": read + write, "read_bytes_per_launch": read, "write_bytes_per_launch": write,
           "fetch_kib_per_dispatch": f_kib, "write_kib_per_dispatch": w_kib, "dispatches": [nf, nw],
           "copy_calibration": {"bytes": copy_bytes, "fetch_kib": cf_kib, "write_kib": cw_kib,
                                "fetch_scale": f_scale, "write_scale": w_scale}}
    path = os.path.join(ROOT, "profiles", "traffic_%s_%s.json" % (args.pmc_call, args.pmc_workload))
    json.dump(out, open(path, "w"), indent=1)
    print(json.dumps(out))


MFMA_PEAK = {"f32": 157.3, "bf16": 2516.6}


def mfma_workload(args, torch, gsm):
    """One step of the large (fp32) or binary (fp32) workload through the
    separate calls; per-call HIP events on the launch stream give each
    kernel's time and the dominant one goes into the roofline entry
    (matrix-core bound)."""
    w = wl.WORKLOADS[args.workload]
    dev = torch.device("cuda:0")
    log("%s: codebook %d x %d, compress" % (w.name, w.Ms[0], w.D))
    C = torch.from_numpy(wl.codebook(w)).to(dev)
    dt = torch.float32
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    Q, R, r, kept, cnorm = gsm.gs_compress(C, q_dtype=dt, r_dtype=dt)
    torch.cuda.synchronize()
    compress_ms = (time.perf_counter() - t0) * 1e3
    B, D, M = w.B, w.D, w.Ms[0]
    # matrices with 16-byte aligned rows, as the library's own outputs are
    rows = lambda n, c, t: gsm.alloc_rows(n, c, t, dev)
    calls = []
    if args.workload == "large":
        P = wl.device_dirichlet_half(B, M, w.seed, torch, dev, dtype=dt)
        X = wl.device_noisy_queries(P, C, w.noise_var, w.seed, torch, dtype=dt)
        T = rows(B, r, dt)
        xn = torch.empty(B, dtype=torch.float32, device=dev)
        S = torch.empty((B, M), dtype=torch.float32, device=dev)
        A = torch.empty((B, M), dtype=torch.float32, device=dev)
        idx = torch.empty(B, dtype=torch.int32, device=dev)
        calls.append(("project", lambda: gsm.gs_project(X, Q, out=T, xnorm2=True, xnorm2_out=xn), 2.0 * B * D * r))
        calls.append(("similarity", lambda: gsm.gs_similarity(T, R, qnorm2=xn, cnorm=cnorm, out=S, argmax_out=idx,
                                                              echelon=True), 2.0 * B * M * r))
        calls.append(("attention", lambda: gsm.gs_attention(T, R, qnorm2=xn, cnorm=cnorm, beta=args.beta, out=A,
                                                            echelon=True), 2.0 * B * M * r))
    else:   # binary: bind pairs
        Pa = torch.from_numpy(wl.probabilities(w, 0)).to(dev)
        Pb = torch.from_numpy(wl.probabilities(w, 0, stream=wl.STREAM_PROBS_B)).to(dev)
        Ta = rows(B, r, torch.float32)
        Tb = rows(B, r, torch.float32)
        S = torch.empty((B, M), device=dev)
        idx = torch.empty(B, dtype=torch.int32, device=dev)
        Y = rows(B, D, torch.float32)
        Ty = rows(B, r, torch.float32)
        calls.append(("prob2vec", lambda: (gsm.gs_prob2vec(Pa, R, out=Ta, echelon=True),
                                           gsm.gs_prob2vec(Pb, R, out=Tb, echelon=True)), 2 * 2.0 * B * M * r))
        calls.append(("similarity", lambda: gsm.gs_similarity(Ta, R, cnorm=cnorm, out=S, argmax_out=idx,
                                                              echelon=True), 2.0 * B * M * r))
        calls.append(("reconstruct_bind", lambda: gsm.gs_reconstruct(Ta, Q, T2=Tb, bind="mul", out=Y),
                      4.0 * B * r * D))
        calls.append(("reproject", lambda: gsm.gs_project(Y, Q, out=Ty), 2.0 * B * D * r))
    stream = torch.cuda.current_stream()
    log("%s: inputs ready (rank %d), %d warm-up step(s)" % (w.name, r, max(1, args.warmup)))
    for _ in range(max(1, args.warmup)):
        for _, f, _ in calls:
            f()
    torch.cuda.synchronize()
    log("%s: %d timed step(s)" % (w.name, args.steps))
    per = {n: [] for n, _, _ in calls}
    evs = []
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        for n, f, _ in calls:
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            f()
            e1.record(stream)
            evs.append((n, e0, e1))
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    for n, e0, e1 in evs:
        per[n].append(e0.elapsed_time(e1))
    flops = {n: fl for n, _, fl in calls}
    # products with the lower-echelon R: flops on its nonzero entries only
    # (2 B nnz(R) per product; R's zero blocks are skipped by the kernels)
    nnz = int((R != 0).sum().item())
    useful = {n: flops[n] * nnz / (M * r) for n in flops if n in ("prob2vec", "similarity", "attention")}
    dom = max(per, key=lambda n: sum(per[n]))
    dom_ms = float(np.mean(per[dom]))
    peak = MFMA_PEAK["f32"]
    achieved = flops[dom] / (dom_ms * 1e-3) / 1e12
    kernel = {"project": "gemm256_store_kernel (X Q^T)", "reproject": "gemm256_store_kernel (Y Q^T)",
              "reconstruct_bind": "gemm256_store_kernel x 2 (T Q, then .* T2 Q)",
              "prob2vec": "gemm256_store_kernel (P R)", "similarity": "similarity scores",
              "attention": "attention weights"}[dom]
    extra_binary = {}
    if args.workload == "binary":
        extra_binary = binary_extras(args, torch, gsm, Pa, R, Ta, Y, per, stream)
    cpu = None
    if not args.no_cpu:
        n = min(args.cpu_rows, B)
        sample = np.sort(np.random.default_rng(w.seed).choice(B, size=n, replace=False))
        si = torch.from_numpy(sample).to(dev)
        if args.workload == "large":
            cpu = cpu_baseline_rows(w, {"X": X.index_select(0, si).cpu().numpy()}, args.beta)
        else:
            cpu = cpu_baseline_rows(w, {"Pa": Pa.index_select(0, si).cpu().numpy(),
                                        "Pb": Pb.index_select(0, si).cpu().numpy()}, args.beta)
    out = {
        "metric": METRIC, "value": B * args.steps / wall, "unit": "queries/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": wall * 1e3 / args.steps,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "f32", "data": "synthetic",
        "config": {"workload": "%s: codebook M=%d, D=%d (r=%d), batch %d; calls %s"
                               % (w.name, M, D, r, B, ", ".join(n for n, _, _ in calls))},
        "roofline": {"bound": "mfma", "kernel": kernel, "call": dom, "achieved": achieved, "peak": peak,
                     "unit": "TFLOP/s", "frac": achieved / peak, "traffic": load_traffic(dom, w.name),
                     "flops_per_launch": flops[dom], "avg_launch_ms": dom_ms},
        "cpu_baseline": cpu,
        "extra": {"per_call_ms": {n: float(np.mean(v)) for n, v in per.items()},
                  "per_call_TFLOPs": {n: flops[n] / (float(np.mean(per[n])) * 1e-3) / 1e12 for n in per},
                  "per_call_useful_TFLOPs": {n: useful[n] / (float(np.mean(per[n])) * 1e-3) / 1e12 for n in useful},
                  "nnz_R": nnz,
                  "compress_ms": compress_ms, "rank": r, "kernel_source_hash": kernel_source_hash(),
                  **extra_binary},
    }
    print(json.dumps(out), flush=True)


def event_ms(torch, f, reps=20):
    """Mean device time of f over reps calls (HIP events on the current stream)."""
    stream = torch.cuda.current_stream()
    for _ in range(3):
        f()
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(reps):
        f()
    e1.record(stream)
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / reps


def binary_extras(args, torch, gsm, Pa, R, Ta, Y, per, stream):
    """Binary workload, two measured side questions.
    1. Sparse probability rows: gs_prob2vec_sparse on the rows truncated to
       the entries above 1e-9 (dropped mass at fp32 level) and to the 16
       largest entries, against the dense product on the full rows.
    2. Fusing restore -> bind -> re-project into one product would keep the
       bound vectors Y on chip: the most it can save is Y's write and re-read,
       timed here as a device copy of Y (read + write of the same bytes)."""
    B, M = Pa.shape
    out = {}
    dense_ms = event_ms(torch, lambda: gsm.gs_prob2vec(Pa, R, out=Ta, echelon=True))
    sp = {"dense_prob2vec_ms": dense_ms}
    Tref = gsm.gs_prob2vec(Pa, R, echelon=True)
    for name in ("above_1e-9", "top16"):
        if name == "top16":
            v, idx = torch.topk(Pa, 16, dim=1)
            idx, order = torch.sort(idx, dim=1)
            v = torch.gather(v, 1, order)
            mask = torch.zeros_like(Pa, dtype=torch.bool).scatter_(1, idx, True)
        else:
            mask = Pa > 1e-9
        counts = mask.sum(dim=1)
        rowptr = torch.zeros(B + 1, dtype=torch.int64, device=Pa.device)
        rowptr[1:] = torch.cumsum(counts, 0)
        cols = torch.nonzero(mask)[:, 1].to(torch.int32).contiguous()
        vals = Pa[mask].contiguous()
        Ts = gsm.alloc_rows(B, R.shape[1], torch.float32, Pa.device)
        ms = event_ms(torch, lambda: gsm.gs_prob2vec_sparse(rowptr, cols, vals, R, out=Ts))
        dropped = (Pa * (~mask)).sum(dim=1)
        err = ((Ts - Tref).abs().max(dim=1).values / Tref.abs().max(dim=1).values.clamp_min(1e-30)).max().item()
        sp[name] = {"ms": ms, "speedup_vs_dense": dense_ms / ms, "nnz_per_row": float(counts.float().mean().item()),
                    "dropped_mass_max": float(dropped.max().item()), "rowrel_diff_vs_full_rows": err}
    out["sparse_prob2vec"] = sp
    Y2 = torch.empty_like(Y)
    copy_ms = event_ms(torch, lambda: Y2.copy_(Y))
    chain = float(np.mean(per["reconstruct_bind"])) + float(np.mean(per["reproject"]))
    out["fused_restore_bind_reproject"] = {
        "y_bytes": Y.numel() * Y.element_size(), "y_round_trip_ms": copy_ms,
        "chain_ms": chain, "max_saving_frac": copy_ms / chain}
    del Y2
    return out


def cpu_baseline_rows(w, inputs, beta):
    """The oracle on a seeded sample of the large or binary batch.  large: cosine
    similarity of x with the codebook, argmax and softmax (project +
    similarity + attention).  binary: v_a = p_a C and v_b = p_b C (prob2vec),
    the cosine similarity of v_a with the codebook and argmax, and the bound
    vector v_a .* v_b (reconstruct + bind); the re-projection is left out
    (the dense side has no basis)."""
    import oracle
    flags = oracle.use_native_build()
    C = wl.codebook(w)
    t0 = time.perf_counter()
    if "X" in inputs:
        n = inputs["X"].shape[0]
        S = oracle.similarity(inputs["X"], C, oracle.COSINE)
        oracle.argmax(S)
        oracle.softmax(S, beta)
        what = "dense fp64 cosine similarity of x with the codebook, argmax, softmax(beta=%g)" % beta
    else:
        n = inputs["Pa"].shape[0]
        Va = oracle.prob2vec(inputs["Pa"], C)
        Vb = oracle.prob2vec(inputs["Pb"], C)
        S = oracle.similarity(Va, C, oracle.COSINE)
        oracle.argmax(S)
        oracle.bind(Va, Vb)
        what = "dense fp64 v = p C for both operands, cosine similarity + argmax, v_a .* v_b"
    dt = time.perf_counter() - t0
    rate = n / dt
    return {"value": rate, "unit": "queries/s", "cores": oracle.threads(), "cpu_model": cpu_model(),
            "kind": "oracle", "build": flags,
            "sample": "%d seeded rows of the %d-row batch: %s; %.1f s; full batch extrapolated to %.0f s"
                      % (n, w.B, what, dt, w.B / rate)}


def cpu_baseline_stress(w, Ps, Xs, beta, rows_desc):
    """The oracle (dense fp64 in D-space) on a seeded sample of the stress
    batch: for each sampled query, cosine similarity of x against every
    codebook vector (what project + similarity compute), argmax, the softmax
    of beta times the scores (attention) and v = p C (what prob2vec +
    reconstruct compute).  Inputs are read back from the device (bf16, upcast
    exactly) before the timed region."""
    import oracle
    flags = oracle.use_native_build()
    C = wl.codebook(w)
    # the natively built copy computes bit for bit what the tested build does
    # (same source, no FMA contraction, no reassociation): checked on two rows
    t0 = time.perf_counter()
    S = oracle.similarity(Xs, C, oracle.COSINE)
    idx = oracle.argmax(S)
    A = oracle.softmax(S, beta)
    V = oracle.prob2vec(Ps, C)
    dt = time.perf_counter() - t0
    n = Xs.shape[0]
    rate = n / dt
    return {"value": rate, "unit": "queries/s", "cores": oracle.threads(), "cpu_model": cpu_model(),
            "kind": "oracle", "build": flags,
            "sample": "%d seeded rows (%s) of the %d-row batch: dense fp64 cosine similarity of x with the "
                      "%d x %d codebook, argmax, softmax(beta=%g), v = p C; %.1f s; full batch extrapolated "
                      "to %.0f s" % (n, rows_desc, w.B, w.Ms[0], w.D, beta, dt, w.B / rate)}, (S, idx, A, V)


def rowrel(g, o):
    """Row-scaled maximum relative difference: max over rows of
    max_j |g - o| / max_j |o|."""
    g = np.asarray(g, np.float64)
    o = np.asarray(o, np.float64)
    den = np.maximum(np.abs(o).max(axis=1), 1e-30)
    return float((np.abs(g - o).max(axis=1) / den).max())


def oracle_check(gpu, ref, tol=2e-2):
    """The step's outputs on the oracle's sample rows against the oracle's
    dense results (taken outside the timed region): row-scaled relative
    differences of S, A and the restored v, and the argmax agreement; an
    argmax differing where the oracle's top two scores are more than twice
    the bf16 tolerance apart would be a fault."""
    Sg, ig, Ag, Vg = gpu
    So, io, Ao, Vo = ref
    srt = np.sort(So, axis=1)
    gap = srt[:, -1] - srt[:, -2]
    band = 2 * tol * np.abs(So).max(axis=1)
    diff = np.asarray(ig) != np.asarray(io)
    return {"rows": int(len(So)), "max_rowrel_S": rowrel(Sg, So), "max_rowrel_A": rowrel(Ag, Ao),
            "max_rowrel_restore": rowrel(Vg, Vo), "tolerance": tol,
            "argmax_differ": int(diff.sum()), "argmax_differ_outside_band": int((diff & (gap > band)).sum()),
            "against": "dense fp64 D-space definitions on the fp32 codebook and the queries' bf16 values"}


def stress_workload(args, torch, gsm):
    """The headline: one step = project, prob2vec, similarity + argmax and
    attention (one score product for both), and reconstruct over the whole
    stress batch (bf16 storage, fp32 accumulation), K steps timed on the synchronised wall clock with HIP
    events around every call."""
    w = wl.WORKLOADS["stress"]
    dev = torch.device("cuda:0")
    B, D, M = w.B, w.D, w.Ms[0]
    dt = torch.bfloat16
    log("stress: codebook %d x %d, compress" % (M, D))
    C = torch.from_numpy(wl.codebook(w)).to(dev)
    # the first call also loads the library's kernels; the second is the
    # steady-state time
    compress_runs = []
    for _ in range(2):
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        Q, R, r, kept, cnorm = gsm.gs_compress(C, q_dtype=dt, r_dtype=dt)
        torch.cuda.synchronize()
        compress_runs.append((time.perf_counter() - t0) * 1e3)
    compress_ms = compress_runs[-1]
    rows = lambda n, c, t: gsm.alloc_rows(n, c, t, dev)
    P = wl.device_dirichlet_half(B, M, w.seed, torch, dev, dtype=dt)
    X = wl.device_noisy_queries(P, C, w.noise_var, w.seed, torch, dtype=dt)
    del C
    T = rows(B, r, dt)
    T2 = rows(B, r, dt)
    xn = torch.empty(B, dtype=torch.float32, device=dev)
    S = torch.empty((B, M), dtype=torch.float32, device=dev)
    A = torch.empty((B, M), dtype=torch.float32, device=dev)
    idx = torch.empty(B, dtype=torch.int32, device=dev)
    Xr = rows(B, D, dt)
    beta = args.beta
    fl_proj, fl_code = 2.0 * B * D * r, 2.0 * B * M * r
    calls = [
        ("project", lambda: gsm.gs_project(X, Q, out=T, xnorm2=True, xnorm2_out=xn), fl_proj),
        ("prob2vec", lambda: gsm.gs_prob2vec(P, R, out=T2, echelon=True), fl_code),
        # the scores once: S, their row argmax and A = softmax(beta S)
        ("similarity_attention", lambda: gsm.gs_similarity_attention(T, R, qnorm2=xn, cnorm=cnorm, beta=beta,
                                                                     out=S, argmax_out=idx, a_out=A,
                                                                     echelon=True), fl_code),
        ("reconstruct", lambda: gsm.gs_reconstruct(T2, Q, out=Xr), fl_proj),
    ]
    stream = torch.cuda.current_stream()
    log("stress: inputs ready (rank %d), %d warm-up step(s)" % (r, args.warmup))
    for _ in range(args.warmup):
        for _, f, _ in calls:
            f()
    torch.cuda.synchronize()
    log("stress: %d timed step(s)" % args.steps)
    evs = []
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        for n, f, _ in calls:
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            f()
            e1.record(stream)
            evs.append((n, e0, e1))
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    per = {n: [] for n, _, _ in calls}
    for n, e0, e1 in evs:
        per[n].append(e0.elapsed_time(e1))
    mean = {n: float(np.mean(v)) for n, v in per.items()}
    flops = {n: fl for n, _, fl in calls}
    # the products with the lower-echelon R skip its zero blocks: also the
    # rate on R's nonzero entries (2 nnz(R) flops per row)
    nnz = int((R != 0).sum().item())
    useful = {n: flops[n] * nnz / (M * r) for n in ("prob2vec", "similarity_attention")}
    dom = max(mean, key=mean.get)
    kernels = {"project": "gemm256_store_kernel<bf16, bf16, BNN=false> (X Q^T, with ||x||^2)",
               "reconstruct": "gemm256_store_kernel<bf16, bf16, BNN=true> (T Q, persistent tile walk)",
               "prob2vec": "gemm256_store_kernel<bf16, bf16, BNN=true> (P R, echelon K ranges)",
               "similarity_attention": "scores256_kernel + rows_sim_attn_reg_kernel<8> (S, argmax, A)"}
    achieved = flops[dom] / (mean[dom] * 1e-3) / 1e12
    peak = MFMA_PEAK["bf16"]
    ms_per_step = wall * 1e3 / args.steps

    # oracle sample rows, read back before anything else is freed
    cpu = None
    if not args.no_cpu:
        n = min(args.cpu_rows, B)
        rng = np.random.default_rng(w.seed)
        sample = np.sort(rng.choice(B, size=n, replace=False))
        si = torch.from_numpy(sample).to(dev)
        Ps = P.index_select(0, si).float().cpu().numpy()
        Xs = X.index_select(0, si).float().cpu().numpy()
        gpu_rows = (S.index_select(0, si).cpu().numpy(), idx.index_select(0, si).cpu().numpy(),
                    A.index_select(0, si).cpu().numpy(), Xr.index_select(0, si).float().cpu().numpy())
    del X, Xr, P, T, T2, S, A, Q, R
    torch.cuda.empty_cache()
    extra = {"per_call_ms": mean,
             "per_call_median_ms": {n: float(np.median(v)) for n, v in per.items()},
             "per_call_min_ms": {n: float(np.min(v)) for n, v in per.items()},
             "per_call_sum_ms": float(sum(mean.values())),
             "per_call_TFLOPs": {n: flops[n] / (mean[n] * 1e-3) / 1e12 for n in mean},
             "per_call_frac_bf16_peak": {n: flops[n] / (mean[n] * 1e-3) / 1e12 / peak for n in mean},
             "per_call_useful_TFLOPs": {n: useful[n] / (mean[n] * 1e-3) / 1e12 for n in useful},
             "nnz_R": nnz, "compress_ms": compress_ms, "compress_first_call_ms": compress_runs[0], "rank": r,
             "timing": "K steps of the four calls on the current stream; HIP events around every call (mean, median and minimum per call)",
             "kernel_source_hash": kernel_source_hash()}
    if not args.no_vsa:
        log("vsa: fused soft selection (both forms)")
        extra["vsa_fused"] = vsa_fused_extra(args, torch, gsm)
    if not args.no_cpu:
        log("oracle: %d sampled rows" % n)
        cpu, ref = cpu_baseline_stress(w, Ps, Xs, beta, "numpy default_rng(%d).choice without replacement" % w.seed)
        extra["oracle_check"] = oracle_check(gpu_rows, ref)
    out = {
        "metric": METRIC, "value": B * args.steps / wall, "unit": "queries/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms_per_step,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16", "data": "synthetic",
        "config": {"workload": "stress: bipolar codebook M=%d (205 duplicated rows, rank %d), D=%d; %d queries "
                               "x = p C + N(0, 0.1), p ~ Dir(1/2); bf16 storage, fp32 accumulation; step = "
                               "project (+||x||^2), prob2vec (echelon R), cosine similarity + argmax and attention "
                               "softmax(beta=%g) from one score product, reconstruct; compress once before timing"
                               % (M, r, D, B, beta),
                   "M": M, "D": D, "rank": r, "batch": B},
        "roofline": {"bound": "mfma", "kernel": kernels[dom], "call": dom, "achieved": achieved, "peak": peak,
                     "unit": "TFLOP/s", "frac": achieved / peak, "traffic": load_traffic(dom, "stress"),
                     "flops_per_launch": flops[dom], "avg_launch_ms": mean[dom]},
        "cpu_baseline": cpu,
        "extra": extra,
    }
    print(json.dumps(out), flush=True)


def memory_workload(args, torch, gsm):
    """Peak device memory of each workload's operators run in D-space on the
    dense codebook against the same outputs through Gram-Space (the paper's
    memory comparison, Sec. 4.2, measured in a run of its own, apart from
    the timing).  Both paths use this library's kernels: the dense path calls
    them with the codebook C itself in place of (Q, R) (r = D: t = p C is
    then the dense vector).  The codebook (C, or Q and R) is built before
    the peak counter is reset and counted separately; peaks are
    torch.cuda.max_memory_allocated over the operators."""
    dev = torch.device("cuda:0")
    rows = lambda n, c, t: gsm.alloc_rows(n, c, t, dev)
    nb = lambda *ts: int(sum(t.numel() * t.element_size() for t in ts if t is not None))
    results = []

    def measure(name, path, codebook, fn):
        torch.cuda.synchronize()
        torch.cuda.empty_cache()
        base = torch.cuda.memory_allocated()
        torch.cuda.reset_peak_memory_stats()
        keep = fn()
        torch.cuda.synchronize()
        peak = torch.cuda.max_memory_allocated() - base
        results.append({"workload": name, "path": path, "codebook_bytes": nb(*codebook), "peak_bytes": int(peak),
                        "outputs_bytes": nb(*keep)})
        log("memory %s %s: codebook %.1f MB, operators peak %.1f MB" % (name, path, nb(*codebook) / 1e6,
                                                                         peak / 1e6))
        del keep

    beta = args.beta
    # vsa: four attribute codebooks, fused soft selection against dense vectors
    w = wl.WORKLOADS["vsa"]
    books = []
    for i, M in enumerate(w.Ms):
        C = torch.from_numpy(wl.codebook(w, i)).to(dev)
        Q, R, r, kept, cn = gsm.gs_compress(C, q_dtype=torch.float32, r_dtype=torch.float32)
        books.append((C, R.contiguous(), cn, torch.from_numpy(wl.probabilities(w, i)).to(dev)))

    def vsa_dense():
        out = []
        for C, R, cn, P in books:
            V = gsm.gs_prob2vec(P, C)                       # dense v = p C, B x D
            S, idx = gsm.gs_similarity(V, C, mode="cosine")
            A, _ = gsm.gs_attention(V, C, mode="cosine", beta=beta)
            del V
            out += [S, idx, A]
        return out

    def vsa_gram():
        groups = [{"P": P, "R": R, "cnorm": cn, "S": torch.empty(P.shape, device=dev),
                   "argmax": torch.empty(P.shape[0], dtype=torch.int32, device=dev),
                   "A": torch.empty(P.shape, device=dev)} for C, R, cn, P in books]
        gsm.gs_soft_select(groups, mode="cosine", beta=beta, form="gram")
        return [t for g in groups for t in (g["S"], g["argmax"], g["A"])]

    measure("vsa", "dense", [b[0] for b in books], vsa_dense)
    measure("vsa", "gram", [b[1] for b in books] + [b[2] for b in books], vsa_gram)
    del books

    # large: hard-selection queries against the codebook
    w = wl.WORKLOADS["large"]
    C = torch.from_numpy(wl.codebook(w)).to(dev)
    Q, R, r, kept, cn = gsm.gs_compress(C, q_dtype=torch.float32, r_dtype=torch.float32)
    P = wl.device_dirichlet_half(w.B, w.Ms[0], w.seed, torch, dev)
    X = rows(w.B, w.D, torch.float32)
    X.copy_(wl.device_noisy_queries(P, C, w.noise_var, w.seed, torch))
    del P
    Cd = rows(C.shape[0], C.shape[1], torch.float32)
    Cd.copy_(C)

    def large_dense():
        S, idx = gsm.gs_similarity(X, Cd, mode="cosine")
        A, _ = gsm.gs_attention(X, Cd, mode="cosine", beta=beta)
        return [S, idx, A]

    def large_gram():
        T, xn = gsm.gs_project(X, Q, xnorm2=True)
        S, idx = gsm.gs_similarity(T, R, qnorm2=xn, cnorm=cn, echelon=True)
        A, _ = gsm.gs_attention(T, R, qnorm2=xn, cnorm=cn, beta=beta, echelon=True)
        return [S, idx, A]

    measure("large", "dense", [Cd], large_dense)
    measure("large", "gram", [Q, R], large_gram)
    del X, C, Cd, Q, R

    # binary: superposition, lookup, bind of restored pairs, re-projection
    w = wl.WORKLOADS["binary"]
    C = torch.from_numpy(wl.codebook(w)).to(dev)
    Q, R, r, kept, cn = gsm.gs_compress(C, q_dtype=torch.float32, r_dtype=torch.float32)
    Pa = torch.from_numpy(wl.probabilities(w, 0)).to(dev)
    Pb = torch.from_numpy(wl.probabilities(w, 0, stream=wl.STREAM_PROBS_B)).to(dev)
    Cd = rows(C.shape[0], C.shape[1], torch.float32)
    Cd.copy_(C)

    def binary_dense():
        Va = gsm.gs_prob2vec(Pa, Cd)
        Vb = gsm.gs_prob2vec(Pb, Cd)
        S, idx = gsm.gs_similarity(Va, Cd, mode="cosine")
        Y = gsm.gs_bind_restored(Va, Vb, op="mul")
        return [S, idx, Y]

    def binary_gram():
        Ta = gsm.gs_prob2vec(Pa, R, echelon=True)
        Tb = gsm.gs_prob2vec(Pb, R, echelon=True)
        S, idx = gsm.gs_similarity(Ta, R, cnorm=cn, echelon=True)
        Y = gsm.gs_reconstruct(Ta, Q, T2=Tb, bind="mul")
        Ty = gsm.gs_project(Y, Q)
        return [S, idx, Y, Ty]

    measure("binary", "dense", [Cd], binary_dense)
    measure("binary", "gram", [Q, R], binary_gram)
    del C, Cd, Q, R, Pa, Pb

    # stress: the full pipeline in bf16
    w = wl.WORKLOADS["stress"]
    dt = torch.bfloat16
    C = torch.from_numpy(wl.codebook(w)).to(dev)
    Q, R, r, kept, cn = gsm.gs_compress(C, q_dtype=dt, r_dtype=dt)
    P = wl.device_dirichlet_half(w.B, w.Ms[0], w.seed, torch, dev, dtype=dt)
    X = wl.device_noisy_queries(P, C, w.noise_var, w.seed, torch, dtype=dt)
    Cd = rows(C.shape[0], C.shape[1], dt)
    Cd.copy_(C)
    del C

    def stress_dense():
        V = gsm.gs_prob2vec(P, Cd)                          # dense superposed vectors, B x D bf16
        S, idx = gsm.gs_similarity(X, Cd, mode="cosine")
        A, _ = gsm.gs_attention(X, Cd, mode="cosine", beta=beta)
        return [V, S, idx, A]

    def stress_gram():
        T, xn = gsm.gs_project(X, Q, out_dtype=dt, xnorm2=True)
        T2 = gsm.gs_prob2vec(P, R, out_dtype=dt, echelon=True)
        S, idx = gsm.gs_similarity(T, R, qnorm2=xn, cnorm=cn, echelon=True)
        A, _ = gsm.gs_attention(T, R, qnorm2=xn, cnorm=cn, beta=beta, echelon=True)
        Xr = gsm.gs_reconstruct(T2, Q, out_dtype=dt)         # restored superposed vectors
        return [T2, S, idx, A, Xr]

    measure("stress", "dense", [Cd], stress_dense)
    measure("stress", "gram", [Q, R], stress_gram)
    del X, P, Cd, Q, R
    by = {}
    for e in results:
        by.setdefault(e["workload"], {})[e["path"]] = e
    ratios = {k: {"peak_dense_over_gram": v["dense"]["peak_bytes"] / max(v["gram"]["peak_bytes"], 1),
                  "codebook_dense_over_gram": v["dense"]["codebook_bytes"] / max(v["gram"]["codebook_bytes"], 1)}
              for k, v in by.items()}
    print(json.dumps({"metric": "peak device memory of the operators, dense vs Gram-Space", "unit": "bytes",
                      "results": results, "ratios": ratios, "kernel_source_hash": kernel_source_hash()}),
          flush=True)


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def dimsweep_workload(args, torch, gsm):
    """Similarity query latency against the original vector dimension D (the
    setting of the paper's codebook-latency table, Sec. 4): a global codebook
    of M = 40 bipolar entries (4 attributes x 10 values), D = 256 .. 8192.
    Dense: cosine similarity of D-space queries X against the codebook C (a
    K = D contraction on the same kernels); Gram-Space: the same scores from
    the coordinates T = X Q^T against R (K = rank = 40).  Queries are
    superposed vectors p C, p = softmax(N(0, 2)) over the 40 entries; a single
    lookup (B = 1) and a batch of 65536 (4096 problems x 16 panels).  Also the
    storage of each form: M D values dense, r D + M r compressed."""
    M, Ds, Bs = 40, [256, 512, 1024, 2048, 4096, 8192], [1, 65536]
    reps = max(10, args.steps)
    stream = torch.cuda.current_stream()

    def timed(f, n=20):
        # n calls captured in one HIP graph, so the per-call time is the
        # device's, not the host's submission rate
        for _ in range(3):
            f()
        torch.cuda.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            for _ in range(n):
                f()
        graph.replay()
        torch.cuda.synchronize()
        ts = []
        for _ in range(reps):
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            graph.replay()
            e1.record(stream)
            ts.append((e0, e1))
        torch.cuda.synchronize()
        return float(np.median([a.elapsed_time(b) for a, b in ts])) * 1e3 / n     # us per call

    rows = []
    for D in Ds:
        C = torch.from_numpy(wl.bipolar_codebook(M, D, 6, D)).cuda()
        Q, R, r, kept, cnorm = gsm.gs_compress(C, q_dtype=torch.float32, r_dtype=torch.float32)
        Cd = gsm.alloc_rows(M, D, torch.float32, "cuda")
        Cd.copy_(C)
        Rc = R.contiguous()
        row = {"D": D, "rank": r, "storage_bytes_dense": 4 * M * D, "storage_bytes_gram": 4 * (r * D + M * r),
               "per_vector_ratio": D / r}
        for B in Bs:
            P = torch.from_numpy(wl.softmax_probs(B, M, float(np.sqrt(2.0)), 6, 100 + D)).cuda()
            X = gsm.alloc_rows(B, D, torch.float32, "cuda")
            X.copy_(P @ C)
            T = gsm.gs_project(X, Q)
            S = torch.empty((B, M), device="cuda")
            idx = torch.empty(B, dtype=torch.int32, device="cuda")
            dense = timed(lambda: gsm.gs_similarity(X, Cd, cnorm=cnorm, out=S, argmax_out=idx))
            gram = timed(lambda: gsm.gs_similarity(T, Rc, cnorm=cnorm, out=S, argmax_out=idx))
            row["B%d" % B] = {"dense_us": dense, "gram_us": gram, "speedup": dense / gram}
            del X, T, S, idx, P
        rows.append(row)
        del C, Cd, Q, R, Rc
        torch.cuda.empty_cache()
    big = rows[-1]["B65536"]
    out = {
        "metric": "similarity query latency vs vector dimension (dense D-space vs Gram-Space)",
        "value": big["gram_us"], "unit": "us", "n_gpus": 1, "steps": reps, "warmup": 5,
        "ms_per_step": big["gram_us"] * 1e-3, "higher_is_better": False, "scaling": "weak",
        "vs_baseline": None, "dtype": "f32", "data": "synthetic",
        "timing": "median over replays of a HIP graph of 20 calls",
        "config": {"workload": "dimsweep: global codebook M=40 bipolar, D=256..8192, cosine similarity + "
                               "argmax, batches of 1 and 65536 queries; value: Gram-Space batch latency at D=8192"},
        "roofline": None, "cpu_baseline": None,
        "extra": {"rows": rows, "kernel_source_hash": kernel_source_hash()},
    }
    print(json.dumps(out), flush=True)


def bind_workload(args, torch, gsm):
    """Binding of restored vectors at the binary workload's shape (16384 rows
    of D = 4096, fp32): blockwise circular convolution and correlation over the
    whole row and over 256-value blocks, xor of binary vectors, element-wise
    product.  Per call: HBM bytes read (two operands) and written (one result)
    over the mean time of a HIP graph of 20 calls."""
    B, D = 16384, 4096
    g = torch.Generator(device="cuda")
    g.manual_seed(7)
    X = gsm.alloc_rows(B, D, torch.float32, "cuda")
    Y = gsm.alloc_rows(B, D, torch.float32, "cuda")
    X.copy_(torch.randn((B, D), generator=g, device="cuda"))
    Y.copy_(torch.randn((B, D), generator=g, device="cuda"))
    Z = gsm.alloc_rows(B, D, torch.float32, "cuda")
    stream = torch.cuda.current_stream()
    reps = max(10, min(args.steps, 50))
    calls = [("conv L=4096", "conv", D), ("corr L=4096", "corr", D), ("conv L=256", "conv", 256),
             ("xor", "xor", None), ("mul", "mul", None)]
    nbytes = 3 * B * D * 4
    per = {}
    for name, op, L in calls:
        f = lambda: gsm.gs_bind_restored(X, Y, op=op, L=L, out=Z)
        for _ in range(3):
            f()
        torch.cuda.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            for _ in range(20):
                f()
        graph.replay()
        torch.cuda.synchronize()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(reps):
            graph.replay()
        e1.record(stream)
        torch.cuda.synchronize()
        us = e0.elapsed_time(e1) * 1e3 / (reps * 20)
        per[name] = {"us": us, "GBps": nbytes / us * 1e-3, "frac": nbytes / us * 1e-3 / HBM_PEAK_GBS}
    dom = "conv L=4096"
    out = {
        "metric": "binding of restored vectors: HBM GB/s vs peak", "value": per[dom]["GBps"], "unit": "GB/s",
        "n_gpus": 1, "steps": reps * 20, "warmup": 3, "ms_per_step": per[dom]["us"] * 1e-3,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32", "data": "synthetic",
        "config": {"workload": "bind: 16384 restored rows of D=4096 (fp32), operators conv / corr (blocks of 4096 "
                               "and 256), xor, mul; value: circular convolution over whole rows"},
        "roofline": {"bound": "hbm", "kernel": "circular_kernel", "call": "gs_bind_restored (conv, L=4096)",
                     "achieved": per[dom]["GBps"], "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": per[dom]["frac"], "traffic": load_traffic("circular_kernel", "bind"),
                     "bytes_per_launch": nbytes,
                     "avg_launch_us": per[dom]["us"]},
        "cpu_baseline": None,
        "extra": {"per_call": per, "bind_coords": bind_coords_extra(torch, gsm, reps),
                  "kernel_source_hash": kernel_source_hash()},
    }
    print(json.dumps(out), flush=True)


def bind_coords_extra(torch, gsm, reps):
    """Restore -> bind -> re-project of coordinate pairs, Z = ((T Q) .* (T2 Q)) Q^T:
    gs_bind_coords (one pass, the bound vectors kept on chip) against the two
    calls gs_reconstruct(bind='mul') + gs_project (B x D written and read
    back), at the large workload's shape (65536 rows, D = 8192, fp32) for
    r = 32 .. 256; mean device time of `reps` calls each (HIP events)."""
    B, D = 65536, 8192
    g = torch.Generator(device="cuda")
    g.manual_seed(11)
    res = {}
    stream = torch.cuda.current_stream()

    def timed(f):
        f()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(reps):
            f()
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / reps
    X = gsm.alloc_rows(B, D, torch.float32, "cuda")
    for r in (32, 64, 128, 256):
        q, _ = torch.linalg.qr(torch.randn((D, r), generator=g, device="cuda"))
        Q = gsm.alloc_rows(r, D, torch.float32, "cuda")
        Q.copy_(q.T)
        T = gsm.alloc_rows(B, r, torch.float32, "cuda")
        T2 = gsm.alloc_rows(B, r, torch.float32, "cuda")
        T.copy_(torch.randn((B, r), generator=g, device="cuda"))
        T2.copy_(torch.randn((B, r), generator=g, device="cuda"))
        Z = gsm.alloc_rows(B, r, torch.float32, "cuda")
        Zc = gsm.alloc_rows(B, r, torch.float32, "cuda")
        fused = timed(lambda: gsm.gs_bind_coords(T, T2, Q, out=Z))
        chain = timed(lambda: (gsm.gs_reconstruct(T, Q, T2=T2, bind="mul", out=X), gsm.gs_project(X, Q, out=Zc)))
        diff = float(((Z - Zc).norm(dim=1) / Zc.norm(dim=1).clamp_min(1e-30)).max().item())
        fl = 3 * 2.0 * B * D * r
        res[str(r)] = {"fused_ms": fused, "two_calls_ms": chain, "speedup": chain / fused,
                       "fused_TFLOPs": fl / fused / 1e9, "fused_frac_f32_peak": fl / fused / 1e9 / MFMA_PEAK["f32"],
                       "max_rowrel_vs_two_calls": diff}
        del Q, T, T2, Z, Zc
    del X
    torch.cuda.empty_cache()
    return {"B": B, "D": D, "per_r": res}


def main():
    args = parse()
    if args.pmc_summary:
        pmc_summary(args)
        return
    if args.gpus != 1:
        print("bench.py measures one GPU: the library has no multi-GPU path (--gpus %d requested)" % args.gpus,
              file=sys.stderr)
        sys.exit(2)
    import torch
    from paper_2608_01528_amd import gramspace as gsm
    global wl
    from paper_2608_01528_amd import workloads as wl_mod
    wl = wl_mod

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    gsm.lib()

    if args.copy_probe_mib:
        n = args.copy_probe_mib * (1 << 20) // 4
        a = torch.ones(n, device="cuda")
        b = torch.empty_like(a)
        for _ in range(5):
            b.copy_(a)
        torch.cuda.synchronize()
        print(json.dumps({"copy_probe_bytes_read": 4 * n, "copy_probe_bytes_written": 4 * n, "launches": 5}))
        return

    if args.workload == "dimsweep":
        dimsweep_workload(args, torch, gsm)
        return
    if args.workload == "bind":
        bind_workload(args, torch, gsm)
        return
    if args.workload == "memory":
        memory_workload(args, torch, gsm)
        return
    if args.workload == "stress":
        stress_workload(args, torch, gsm)
        return
    if args.workload in ("large", "binary"):
        mfma_workload(args, torch, gsm)
        return
    vsa_workload(args, torch, gsm)


def vsa_prepare(args, torch, gsm):
    w = wl.WORKLOADS["vsa"]
    per_set = sum(w.B * (16 * M + 4) for M in w.Ms)
    nsets = args.sets or max(1, int(np.ceil((1 << 30) / per_set)))
    work = VsaWorkload(w, nsets, torch, gsm)
    prepared = []
    for s in range(nsets):
        # the fused step reads P and writes the scores, their argmax and the
        # attention weights; the coordinates are an intermediate
        groups = [{"P": b["sets"][s]["P"], "R": b["R"], "cnorm": b["cnorm"],
                   "S": b["sets"][s]["S"], "argmax": b["sets"][s]["argmax"], "A": b["sets"][s]["A"]}
                  for b in work.books]
        prepared.append(gsm.soft_groups(groups))
    return w, work, nsets, prepared


def vsa_fused_extra(args, torch, gsm, steps=200):
    """The fused soft selection of the vsa workload in both of its forms:
    scores through the Gram matrix (soft_gram_kernel) and through the
    coordinates t = p R formed in registers (soft_select_kernel, T not
    stored).  Each: `steps` launches in one HIP graph, replayed once."""
    w, work, nsets, prepared = vsa_prepare(args, torch, gsm)
    stream = torch.cuda.current_stream()
    bpl = float(work.fused_bytes())
    out = {"workload": "vsa: 4 bipolar attribute codebooks M=5,6,10,22, D=1024; 65536 probability rows each "
                       "(262144 queries per launch); fp32; cosine similarity + argmax + softmax(beta=%g); "
                       "%d batch copies (>= 1 GiB) cycled" % (args.beta, nsets),
           "bytes_per_launch": bpl, "compress_ms": work.compress_ms}
    for form, kernel in (("gram", "soft_gram_kernel"), ("coords", "soft_select_kernel")):
        def step(k, form=form):
            gsm.gs_soft_select(None, mode="cosine", beta=args.beta, prepared=prepared[k % nsets], form=form)
        for k in range(10):
            step(k)
        torch.cuda.synchronize()
        wall, launch_ms = timed_graph(torch, steps, step, stream)
        gbs = bpl / (launch_ms * 1e-3) / 1e9
        out[form] = {"kernel": kernel, "ms_per_step": wall * 1e3 / steps, "avg_launch_us": launch_ms * 1e3,
                     "queries_per_s": work.queries * steps / wall, "GBps": gbs, "frac_hbm": gbs / HBM_PEAK_GBS,
                     "traffic": load_traffic(kernel, "vsa")}
    del work, prepared
    torch.cuda.empty_cache()
    return out


def vsa_workload(args, torch, gsm):
    """--workload vsa: the fused soft selection (Gram form) as the headline."""
    w, work, nsets, prepared = vsa_prepare(args, torch, gsm)
    beta = args.beta

    def fused_step(k):
        gsm.gs_soft_select(None, mode="cosine", beta=beta, prepared=prepared[k % nsets], form="gram")

    def coords_step(k):
        gsm.gs_soft_select(None, mode="cosine", beta=beta, prepared=prepared[k % nsets], form="coords")

    def unfused_step(k):
        for b in work.books:
            d = b["sets"][k % nsets]
            gsm.gs_prob2vec(d["P"], b["R"], out=d["T"])
            gsm.gs_similarity(d["T"], b["R"], cnorm=b["cnorm"], mode="cosine", out=d["S"], argmax_out=d["argmax"])
            gsm.gs_attention(d["T"], b["R"], cnorm=b["cnorm"], mode="cosine", beta=beta, out=d["A"])

    stream = torch.cuda.current_stream()
    for k in range(args.warmup):
        fused_step(k)
        coords_step(k)
        if not args.no_unfused:
            unfused_step(k)
    torch.cuda.synchronize()

    wall, launch_ms = timed_graph(torch, args.steps, fused_step, stream)
    ms_per_step = wall * 1e3 / args.steps
    qps = work.queries * args.steps / wall
    bpl = float(work.fused_bytes())
    achieved = bpl / (launch_ms * 1e-3) / 1e9

    extra = {
        "timing": "one HIP graph of K fused launches; events on the replay stream",
        "fused_step_bytes": bpl,
        "compress_ms": work.compress_ms,
        "kernel_source_hash": kernel_source_hash(),
        "buffer_copies": nsets,
    }
    cwall, claunch = timed_graph(torch, args.steps, coords_step, stream)
    extra["coords_form"] = {"kernel": "soft_select_kernel", "ms_per_step": cwall * 1e3 / args.steps,
                            "avg_launch_us": claunch * 1e3, "queries_per_s": work.queries * args.steps / cwall,
                            "GBps": bpl / (claunch * 1e-3) / 1e9}
    if args.streams > 1:
        cwall, _ = timed_graph(torch, args.steps, fused_step, stream, nstreams=args.streams)
        extra["concurrent"] = {"streams": args.streams, "ms_per_step": cwall * 1e3 / args.steps,
                               "queries_per_s": work.queries * args.steps / cwall,
                               "GBps": bpl * args.steps / cwall / 1e9}
    if not args.no_unfused:
        uwall, _ = timed_graph(torch, args.steps, unfused_step, stream)
        extra["unfused_12_calls_ms_per_step"] = uwall * 1e3 / args.steps
        extra["unfused_queries_per_s"] = work.queries * args.steps / uwall
        extra["unfused_step_bytes"] = work.unfused_bytes()
        extra["unfused_GBps"] = work.unfused_bytes() / (uwall / args.steps) / 1e9

    # hot-cache reference: the fused step on one batch copy (cache resident)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        for k in range(args.steps):
            gsm.gs_soft_select(None, mode="cosine", beta=beta, prepared=prepared[0], form="gram")
    g.replay()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    g.replay()
    torch.cuda.synchronize()
    extra["hot_cache_ms_per_step"] = (time.perf_counter() - t0) * 1e3 / args.steps

    cpu = None if args.no_cpu else cpu_baseline_vsa(w, beta, args.cpu_seconds)
    out = {
        "metric": METRIC,
        "value": qps,
        "unit": "queries/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {
            "workload": "vsa: 4 bipolar attribute codebooks M=5,6,10,22, D=1024; 4096 problems x 16 panels "
                        "= 65536 probability rows each; prob2vec + cosine similarity/argmax + softmax(beta=%g) "
                        "fused in one launch, scores through the codebook Gram matrix R R^T (no coordinates "
                        "formed); outputs S, argmax, A" % beta,
            "codebooks_M": w.Ms, "D": w.D, "rows_per_codebook": w.B, "queries_per_step": work.queries,
        },
        "roofline": {
            "bound": "hbm", "kernel": "soft_gram_kernel", "call": "gs_soft_select (Gram form)",
            "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": achieved / HBM_PEAK_GBS,
            "traffic": load_traffic("soft_gram_kernel", "vsa"),
            "bytes_per_launch": bpl, "avg_launch_us": launch_ms * 1e3,
        },
        "cpu_baseline": cpu,
        "extra": extra,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
