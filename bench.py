"""Benchmark of the hot path on one MI355X: sparse absorbed-MLA partial
attention of routed query rows over selected 64-token latent blocks, then the
requester-side LSE merge of the partials.

One step = one pass of the whole path over one batch: mla_sparse_partial_attn
over every (request, chunk) job, then mla_merge_partials over each request's
partials.  Default workload: 64 routed requests (Mq = 1, 128 heads), each
hitting 4 chunks of a 256-chunk x 8192-token bf16 pool and selecting 32
blocks (2048 tokens) per chunk -> 256 partials merged into 64 outputs.

Prints one JSON line.  `value` is microseconds per routed request (whole step
/ requests, inputs resident in HBM): K steps are launched back to back on one
stream and timed with HIP events recorded on that stream, so for small steps
the figure includes any time the GPU waits for the host to launch.  The
dominant kernel's roofline uses algorithmic bytes (selected KV + query rows +
partial outputs) over the partial call's time measured the same way;
`cpu_baseline` is the oracle timed on a bounded sample.
"""
import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
BF16_PEAK_TFLOPS = 2500.0
DLAT, DPE, BLOCK = 512, 64, 64


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="batched-merge",
                    help="batched-merge | dsv3-one-request | few-head | dense-local | "
                         "dense-local-fp8 | tiny | holder-{dense|sparse}-n<N>-h<H>[-jobs] "
                         "(one holder chunk serving N requesters) | "
                         "select-{tok|blk|dense}-b<B>-k<k>-c<corpus>[-h<H>] (selection budget) | "
                         "fetch-splice-c<n>-l<L> | fetch-gather-k<k>-c<corpus>-l<L> (FETCH side)")
    ap.add_argument("--n-splits", type=int, default=0, help="split-K override (0 = library)")
    ap.add_argument("--cpu-seconds", type=float, default=15.0,
                    help="target CPU time of the oracle sample (0 = skip)")
    ap.add_argument("--warmup-seconds", type=float, default=1.0,
                    help="extra untimed steps for at least this long, so clocks settle")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="also run one plain device copy of this many MiB (untimed), a "
                         "known-size reference for hardware byte counters")
    ap.add_argument("--cold-reps", type=int, default=-1,
                    help="replica input sets for the cold-cache timing (-1: enough that the "
                         "rotation touches more than 512 MiB, for workloads that touch less "
                         "than 256 MiB per call; 0: skip)")
    return ap.parse_args()


def stats_ms(durations):
    """mean, p50 and min of per-step durations (ms)."""
    d = np.asarray(durations, dtype=np.float64)
    return {"mean": float(d.mean()), "p50": float(np.median(d)), "min": float(d.min())}


def event_times(stream, fns, reps):
    """Run fns[i % len(fns)] reps times back to back on `stream`, with a HIP
    event recorded on that stream between consecutive calls; returns the
    per-call durations in ms."""
    import torch
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(reps + 1)]
    stream.synchronize()
    ev[0].record(stream)
    for i in range(reps):
        fns[i % len(fns)]()
        ev[i + 1].record(stream)
    stream.synchronize()
    return [ev[i].elapsed_time(ev[i + 1]) for i in range(reps)]


def code_fingerprint(path):
    """SHA-256 of a C/HIP source with its comments and white space removed:
    it changes with the code, not with edits of comments."""
    import hashlib
    import re
    with open(path) as f:
        text = f.read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    text = re.sub(r"//[^\n]*", "", text)
    return hashlib.sha256("".join(text.split()).encode()).hexdigest()


def counted_traffic(workload, n_splits, kernel="partial_kernel"):
    """HBM bytes per launch of the kernel from the committed rocprofv3
    counter summary (FETCH_SIZE / WRITE_SIZE scaled by a known-size copy), or
    None when that summary is for another workload or an older kernel source."""
    path = os.path.join(ROOT, "profiles", f"{kernel}_{workload}_counters.json")
    if n_splits != 0 or not os.path.exists(path):
        return None
    with open(path) as f:
        d = json.load(f)
    fp = sources_fingerprint(d.get("sources") or [d["source"]])
    return d["traffic_bytes"] if fp == d.get("source_code_fingerprint") else None


def counted_flop(workload, n_splits):
    """Matrix-core FLOP per launch of the partial kernel from the committed
    rocprofv3 counter summary (SQ_INSTS_VALU_MFMA_MOPS_BF16 x 512), or None
    when there is none for this workload or it is for an older source."""
    path = os.path.join(ROOT, "profiles", f"partial_kernel_{workload}_mfma.json")
    if n_splits != 0 or not os.path.exists(path):
        return None
    with open(path) as f:
        d = json.load(f)
    fp = sources_fingerprint(d["sources"])
    return d["flop_per_dispatch"] if fp == d.get("source_code_fingerprint") else None


def sources_fingerprint(sources):
    """code_fingerprint of one source, or of several (the kernel's file and
    the headers it includes) combined."""
    fps = [code_fingerprint(os.path.join(ROOT, s)) for s in sources]
    if len(fps) == 1:
        return fps[0]
    import hashlib
    return hashlib.sha256("".join(fps).encode()).hexdigest()


def q_rows(w):
    """The distinct q rows the call is given: a workload whose jobs repeat
    their requests' q (slot-major, job j * n + b reading request b's q)
    passes the first n rows once; any other passes one per job."""
    return int((w.meta or {}).get("q_rows", w.q_lat.shape[0]))


def algorithmic(w):
    """(FLOP, bytes) of one partial-attention launch over workload w."""
    R, Mq, H, _ = w.q_lat.shape
    rows = R * Mq * H
    flops = w.algorithmic_flops()
    kv = w.kv_bytes()  # the selected entries (blocks shared by query rows once)
    # q once per distinct row: jobs that share a request's q read it once
    q = q_rows(w) * Mq * H * (DLAT + DPE) * 2
    out = rows * (DLAT + 1) * 4
    return flops, kv + q + out, kv


def bench_fetch(args):
    """The FETCH-side kernels: the splice of a pulled chunk (every layer, one
    launch) or the gather of a selected token set.  One step = one call."""
    import torch
    from paper_2606_01502_amd import mla, workloads as W
    from tests import gpu_helpers as G

    mla.load()
    w = W.fetch_inputs(args.workload)
    dev = G.device()

    def bf16(a):
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).to(dev)

    def i32(a):
        return torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).to(dev)

    stream = torch.cuda.Stream()
    ckv, kpe, table = bf16(w["ckv"]), bf16(w["kpe"]), i32(w["table"])
    L, n = w["L"], w["n"]
    if w["kind"] == "splice":
        cc, ck = bf16(w["chunk_ckv"]), bf16(w["chunk_kpe"])

        def call():
            mla.fetch_splice(cc, ck, ckv, kpe, table, w["dst_start"], w["delta"], stream=stream)
    else:
        sel = i32(w["sel"])
        oc = torch.empty((L, n, DLAT), dtype=torch.bfloat16, device=dev)
        ok = torch.empty((L, n, DPE), dtype=torch.bfloat16, device=dev)

        def call():
            mla.fetch_gather(ckv, kpe, table, sel, oc, ok, stream=stream)
    torch.cuda.synchronize()
    with torch.cuda.stream(stream):
        for _ in range(args.warmup):
            call()
        stream.synchronize()
        t_w = time.perf_counter()
        while time.perf_counter() - t_w < args.warmup_seconds:
            call()
            stream.synchronize()
        if args.copy_calibration_mib > 0:
            src = torch.ones(args.copy_calibration_mib << 18, dtype=torch.float32, device=dev)
            dst = torch.empty_like(src)
            dst.copy_(src)
            stream.synchronize()
            del src, dst
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        e0.record(stream)
        for _ in range(args.steps):
            call()
        e1.record(stream)
        stream.synchronize()
        t1 = time.perf_counter()
    ms = e0.elapsed_time(e1) / args.steps
    # algorithmic bytes: every token row read once and written once, all layers
    alg_bytes = 2 * L * n * (DLAT + DPE) * 2
    achieved = alg_bytes / (ms * 1e-3) / 1e9
    cpu = None
    if args.cpu_seconds > 0:
        # the oracle on one layer of the same call, scaled to all L layers
        from oracle import fetch as F  # test infrastructure: the CPU baseline only
        ts = time.perf_counter()
        if w["kind"] == "splice":
            F.splice(w["chunk_ckv"][:1], w["chunk_kpe"][:1], w["ckv"][:1], w["kpe"][:1],
                     w["table"], w["dst_start"], w["delta"], 10000.0, 0)
        else:
            F.gather(w["ckv"][:1], w["kpe"][:1], w["table"], w["sel"])
        one = time.perf_counter() - ts
        cpu = {"value": one * L * 1e6, "unit": "us/call", "cores": 1, "kind": "oracle",
               "sample": f"1 of {L} layers, numpy oracle, scaled by {L}"}
    what = "splice of a pulled chunk" if w["kind"] == "splice" else "gather of a selected set"
    kernel = "splice_kernel" if w["kind"] == "splice" else "gather_kernel"
    res = {
        "metric": f"us per FETCH {what} (all layers, one call)",
        "value": ms * 1e3, "unit": "us/call", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms, "higher_is_better": False, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": w["name"], "layers": L, "tokens": n},
        "host_wall_ms_per_step": (t1 - t0) * 1e3 / args.steps,
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBS,
                     "traffic": counted_traffic(w["name"], 0, kernel), "kernel": kernel,
                     "algorithmic_bytes": alg_bytes},
        "cpu_baseline": cpu,
    }
    print(json.dumps(res), flush=True)


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only: this build has no multi-GPU path "
              f"(asked for --gpus {args.gpus})", file=sys.stderr)
        sys.exit(2)
    if args.workload.startswith("fetch-"):
        return bench_fetch(args)

    import torch
    from paper_2606_01502_amd import mla, workloads as W
    from tests import gpu_helpers as G

    mla.load()  # fail loudly before any work if the library is missing
    w = W.make(args.workload)
    R, Mq, H, _ = w.q_lat.shape
    t = G.upload(w)
    dev = G.device()
    out_lat = torch.empty((R, Mq, H, DLAT), dtype=torch.float32, device=dev)
    out_lse = torch.empty((R, Mq, H), dtype=torch.float32, device=dev)
    n_req = w.n_requests
    parts = w.merge_parts
    merged = torch.empty((n_req, Mq, H, DLAT), dtype=torch.float32, device=dev) if parts > 1 else None
    part_lat = [out_lat[j * n_req:(j + 1) * n_req] for j in range(parts)]
    part_lse = [out_lse[j * n_req:(j + 1) * n_req] for j in range(parts)]

    # All work runs on one side stream (default priority).  The calls are
    # prepared once (descriptors built, stream fixed), as a serving loop over
    # static buffers would hold them, so the host side stays ahead of the GPU.
    stream = torch.cuda.Stream()
    # the distinct q rows only (job r reads q row r mod their count)
    n_q = q_rows(w)
    t["q_lat"], t["q_pe"] = t["q_lat"][:n_q], t["q_pe"][:n_q]
    partial = mla.prepare_partial(t["q_lat"], t["q_pe"], t["ckv"], t["kpe"], t["table"],
                                  t["sel"], w.scale, out_lat, out_lse, t["ckv_scale"],
                                  t["kpe_scale"], n_splits=args.n_splits, stream=stream,
                                  tokens=w.tokens)
    merge = (mla.prepare_merge(part_lat, part_lse, out=merged, stream=stream)
             if merged is not None else (lambda: None))
    torch.cuda.synchronize()
    with torch.cuda.stream(stream):
        for _ in range(args.warmup):
            partial()
            merge()
        stream.synchronize()
        t_w = time.perf_counter()
        while time.perf_counter() - t_w < args.warmup_seconds:
            partial()
            merge()
            stream.synchronize()
        if args.copy_calibration_mib > 0:
            n = args.copy_calibration_mib << 18  # float32 elements
            src = torch.ones(n, dtype=torch.float32, device=dev)
            dst = torch.empty_like(src)
            dst.copy_(src)
            stream.synchronize()
            del src, dst

        K = args.steps

        # The timed region: K steps launched back to back on the stream, an
        # event between consecutive steps (per-step p50 and min; the mean is
        # the whole region over K).
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        step_d = event_times(stream, [lambda: (partial(), merge())], K)
        torch.cuda.synchronize()
        t1 = time.perf_counter()
        partial_d = event_times(stream, [partial], K)
        merge_d = event_times(stream, [merge], K) if merged is not None else [0.0]
        # The same step with the partials in Section 3.2's wire form (bf16
        # rows with (m, l), 1032 B per row instead of 2052), as a holder would
        # ship them: reported beside the fp32 step, not as the value.
        wire = None
        if merged is not None:
            w_lat = torch.empty((R, Mq, H, DLAT), dtype=torch.bfloat16, device=dev)
            w_ml = torch.empty((R, Mq, H, 2), dtype=torch.float32, device=dev)
            w_partial = mla.prepare_partial(t["q_lat"], t["q_pe"], t["ckv"], t["kpe"], t["table"],
                                            t["sel"], w.scale, w_lat, w_ml, t["ckv_scale"],
                                            t["kpe_scale"], n_splits=args.n_splits, stream=stream,
                                            tokens=w.tokens, wire=True)
            w_merged = torch.empty_like(merged)
            w_merge = mla.prepare_merge([w_lat[j * n_req:(j + 1) * n_req] for j in range(parts)],
                                        [w_ml[j * n_req:(j + 1) * n_req] for j in range(parts)],
                                        out=w_merged, stream=stream)
            for _ in range(max(args.warmup, 3)):
                w_partial()
                w_merge()
            stream.synchronize()
            wire = {"step_us": {k: v * 1e3 for k, v in stats_ms(
                        event_times(stream, [lambda: (w_partial(), w_merge())], K)).items()},
                    "partial_us": {k: v * 1e3 for k, v in stats_ms(
                        event_times(stream, [w_partial], K)).items()},
                    "merge_us": {k: v * 1e3 for k, v in stats_ms(
                        event_times(stream, [w_merge], K)).items()}}
            stream.synchronize()
            wire["merged_max_row_rel_diff_vs_fp32"] = float(G.row_errors(
                w_merged.cpu().numpy().astype(np.float64),
                merged.cpu().numpy().astype(np.float64)).max())
            del w_lat, w_ml, w_merged
        partial()
        merge()  # leave the outputs of one whole step in place
        torch.cuda.synchronize()
    step_st, partial_st, merge_st = stats_ms(step_d), stats_ms(partial_d), stats_ms(merge_d)
    ms_step = step_st["mean"]
    partial_ms = partial_st["mean"]
    merge_ms = merge_st["mean"]

    # ---- cold caches: the same calls rotating over replica input sets (the
    # same values at other addresses) that together touch more than 512 MiB,
    # more than the 256 MiB last-level cache, so no call finds its inputs
    # cached by the previous ones
    flops, alg_bytes, kv_bytes = algorithmic(w)
    cold = None
    n_rep = args.cold_reps
    if n_rep < 0:
        n_rep = (int((512 << 20) // max(alg_bytes, 1)) + 2) if alg_bytes < (256 << 20) else 0
        n_rep = min(max(n_rep, 8), 4096) if n_rep else 0
        pool_bytes = sum(v.numel() * v.element_size() for v in t.values() if v is not None)
        n_rep = min(n_rep, int(32e9 // max(pool_bytes, 1)))  # replicas of every input
    if n_rep > 0:
        reps = []
        for _ in range(n_rep):
            rt = {k: (v.clone() if v is not None else None) for k, v in t.items()}
            if t["ckv_scale"] is not None and t["kpe_scale"] is t["ckv_scale"]:
                rt["kpe_scale"] = rt["ckv_scale"]
            po = mla.prepare_partial(rt["q_lat"], rt["q_pe"], rt["ckv"], rt["kpe"], rt["table"],
                                     rt["sel"], w.scale, out_lat, out_lse, rt["ckv_scale"],
                                     rt["kpe_scale"], n_splits=args.n_splits, stream=stream,
                                     tokens=w.tokens)
            reps.append((rt, po))
        calls = [r[1] for r in reps]
        with torch.cuda.stream(stream):
            for c in calls:
                c()
            stream.synchronize()
            cold_d = event_times(stream, calls, max(K, 2 * n_rep))
            step_cold_d = event_times(stream, [(lambda c=c: (c(), merge())) for c in calls],
                                      max(K, 2 * n_rep))
            partial()
            merge()
            torch.cuda.synchronize()
        touched = n_rep * alg_bytes
        cold = {"replicas": n_rep, "touched_mib": touched / 2 ** 20,
                "partial_us": {k: v * 1e3 for k, v in stats_ms(cold_d).items()},
                "step_us": {k: v * 1e3 for k, v in stats_ms(step_cold_d).items()},
                "us_per_request_p50": stats_ms(step_cold_d)["p50"] * 1e3 / n_req}
        del reps, calls

    part_s = partial_ms * 1e-3
    achieved = alg_bytes / part_s / 1e9
    tflops = flops / part_s / 1e12
    us_per_req = ms_step * 1e3 / n_req

    # ---- oracle on a bounded sample of the same workload (whole requests)
    cpu = None
    parity = None
    if args.cpu_seconds > 0:
        import oracle  # test infrastructure: timed here as the CPU baseline only
        out_np = out_lat.cpu().numpy()
        lse_np = out_lse.cpu().numpy()
        merged_np = merged.cpu().numpy() if merged is not None else None

        # requesters are jobs (slot-major: hit j of every request, then hit
        # j+1), or the query rows of one job (one holder serving them all)
        rows_are_requests = R == 1 and n_req > 1 and Mq == n_req

        def jobs_of(reqs):
            reqs = np.asarray(reqs)
            if rows_are_requests:
                return (np.zeros(1, np.int64), reqs)
            return (np.concatenate([j * n_req + reqs for j in range(parts)]), slice(None))

        def run_oracle(reqs):
            js, ri = jobs_of(reqs)
            sel = w.sel[js][:, ri] if w.sel.ndim == 3 else w.sel[js]
            return (js, ri), oracle.partial(w.q_lat[js][:, ri], w.q_pe[js][:, ri], w.ckv, w.kpe,
                                            w.table[js], sel, w.scale, w.ckv_scale, w.kpe_scale,
                                            tokens=w.tokens)

        ts = time.perf_counter()
        js, (o1, l1) = run_oracle([0])
        one = time.perf_counter() - ts
        n = int(min(n_req, max(1, round(args.cpu_seconds / max(one, 1e-3)))))
        reqs = list(range(n))
        ts = time.perf_counter()
        js, (o_ref, l_ref) = run_oracle(reqs)
        if parts > 1:
            po = np.stack([o_ref[j * n:(j + 1) * n] for j in range(parts)])
            pl = np.stack([l_ref[j * n:(j + 1) * n] for j in range(parts)])
            m_ref, _ = oracle.merge(po, pl)
        elapsed = time.perf_counter() - ts
        js, ri = js
        cpu = {"value": elapsed * 1e6 / n, "unit": "us/request", "cores": oracle.default_threads(),
               "kind": "oracle",
               "sample": f"{n} of {n_req} requests ({len(js)} of {R} partial jobs"
                         f"{' + their merge' if parts > 1 else ''}), fp64 C oracle"}
        # the same oracle on one host thread, over one request (partials only)
        js1, ri1 = jobs_of([0])
        sel1 = w.sel[js1][:, ri1] if w.sel.ndim == 3 else w.sel[js1]
        ts = time.perf_counter()
        oracle.partial(w.q_lat[js1][:, ri1], w.q_pe[js1][:, ri1], w.ckv, w.kpe, w.table[js1], sel1,
                       w.scale, w.ckv_scale, w.kpe_scale, tokens=w.tokens, n_threads=1)
        cpu["value_1core"] = (time.perf_counter() - ts) * 1e6
        cpu["sample_1core"] = "request 0 (its partial jobs), fp64 C oracle, 1 thread"
        rel = G.row_errors(out_np[js][:, ri].astype(np.float64), o_ref)
        lse_err = np.abs(lse_np[js][:, ri] - l_ref)
        parity = {"rows": int(rel.size), "max_row_rel_err": float(rel.max()),
                  "max_lse_abs_err": float(lse_err[np.isfinite(l_ref)].max())
                  if np.isfinite(l_ref).any() else 0.0}
        if parts > 1:
            parity["merge_max_row_rel_err"] = float(
                G.row_errors(merged_np[:n].astype(np.float64), m_ref).max())

    # The bound is the roofline side the kernel's algorithmic intensity falls
    # on (ridge = bf16 MFMA peak / HBM peak, about 312 FLOP/B).
    traffic = counted_traffic(w.name, args.n_splits)
    c_flop = counted_flop(w.name, args.n_splits)
    common = {"traffic": traffic, "kernel": "partial_kernel", "algorithmic_bytes": alg_bytes,
              "kv_bytes": kv_bytes, "flops": flops,
              "intensity_flop_per_byte": flops / alg_bytes,
              # the matrix core's own count of the work (rocprofv3 counter), per
              # launch, over the same event-timed duration as `achieved`
              "counter_flop": c_flop,
              "counter_tflops": c_flop / (partial_ms * 1e-3) / 1e12 if c_flop else None}
    if flops / alg_bytes > BF16_PEAK_TFLOPS * 1e12 / (HBM_PEAK_GBS * 1e9):
        roofline = {"bound": "mfma", "achieved": tflops, "peak": BF16_PEAK_TFLOPS,
                    "unit": "TFLOP/s", "frac": tflops / BF16_PEAK_TFLOPS, **common}
    else:
        roofline = {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                    "frac": achieved / HBM_PEAK_GBS, **common}

    merge_roofline = None
    if merged is not None:
        m_rows = n_req * Mq * H
        m_bytes = m_rows * (parts * (DLAT + 1) * 4 + DLAT * 4)  # parts + their lse in, rows out
        m_ach = m_bytes / (merge_ms * 1e-3) / 1e9
        m_traffic = counted_traffic(w.name, args.n_splits, "merge_kernel")
        merge_roofline = {"bound": "hbm", "achieved": m_ach, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                          "frac": m_ach / HBM_PEAK_GBS, "traffic": m_traffic,
                          "kernel": "merge_kernel", "algorithmic_bytes": m_bytes}
    res = {
        "metric": "us per routed request (sparse MLA partial attn + LSE merge)",
        "value": us_per_req,
        "unit": "us/request",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "fp8-e4m3 kv, bf16 mfma" if w.fp8 else "bf16",
        "data": "synthetic",
        "device": {"name": torch.cuda.get_device_name(0),
                   "arch": getattr(torch.cuda.get_device_properties(0), "gcnArchName", None),
                   "hip": torch.version.hip},
        "config": {"workload": w.name, "requests": n_req, "jobs": R, "mq": Mq, "heads": H,
                   ("selected_tokens" if w.tokens else "selected_blocks"): int((w.sel >= 0).sum()),
                   "block_tokens": BLOCK,
                   "pool_blocks": int(w.ckv.shape[0]), "merge_parts": parts},
        "tflops": tflops,
        "pct_bf16_mfma_peak": 100.0 * tflops / BF16_PEAK_TFLOPS,
        "partial_kernel_us": partial_ms * 1e3,
        "merge_us": merge_ms * 1e3 if merged is not None else 0.0,
        "step_us": {k: v * 1e3 for k, v in step_st.items()},
        "partial_us": {k: v * 1e3 for k, v in partial_st.items()},
        "merge_us_stats": ({k: v * 1e3 for k, v in merge_st.items()} if merged is not None
                           else None),
        "merge_roofline": merge_roofline,
        "wire_form": wire,
        "cold": cold,
        "host_wall_ms_per_step": (t1 - t0) * 1e3 / K,
        "roofline": roofline,
        "cpu_baseline": cpu,
        "parity_sample": parity,
    }
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
