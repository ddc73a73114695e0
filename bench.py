"""Benchmark of the fused sampling hot path on one MI355X.

Default workload: the heterogeneous singular batch -- B=64 requests,
V=131072 bf16 logits, half greedy, half stochastic with per-request
temperature / top-k / top-p / min-p, repetition / frequency / presence
penalties over a 512-token history and a 16-entry sparse logit bias.
One step = one ss_sample call (streaming kernel + row merge kernel) on one batch.

Timing: the K steps are captured in HIP graphs over R rotated logit buffers
(R x 16.8 MB > 2 x the 256 MB Infinity Cache, so every step reads HBM) and
replayed between two events after warm-up; value = rows / s over the timed
region.  Each kernel's own duration is then measured over a second timed
region of eager steps on the same stream and buffers: the library records
three HIP events per step (before the streaming kernel, between the two
kernels, after the merge kernel; ss_set_kernel_events), with no host sync
inside the loop.  The roofline object describes the kernel with the larger
average duration, its algorithmic bytes per launch over that duration
against 8 TB/s; both kernels' figures are listed under "kernels".

Counter mode (--traffic-from FETCH_DIR WRITE_DIR OUT): reads two rocprofv3
--pmc runs of this script (FETCH_SIZE, then WRITE_SIZE) and writes the HBM
bytes per launch of both kernels, each counter scaled by what it reads for
the 16 MiB device copies this script makes, with the kernel-source hash the
counters belong to.

Prints one JSON line.
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

METRIC = ("µs per batch + rows/sec for fused sample/verify at V=2^17; "
          "achieved HBM GB/s vs peak")
HBM_PEAK_GBS = 8000.0
MALL_BYTES = 256 << 20


def _params_bytes(inp):
    n = 0
    for k in ("mode", "temperature", "top_k", "top_p", "min_p", "rep", "freq", "pres", "seed", "position",
              "hist_offsets", "hist_ids", "bias_offsets", "bias_ids", "bias_vals", "bitmask"):
        a = inp.get(k)
        if a is not None:
            n += np.asarray(a).nbytes
    return n


def algorithmic_bytes(inp, out_bytes_per_row=12):
    """Bytes one pass must move: logits once, sparse lists, params, outputs."""
    logits = np.asarray(inp["x"]).nbytes
    return logits, logits + _params_bytes(inp) + out_bytes_per_row * inp["B"]


def stream_alg_bytes(inp):
    """Streaming kernel: every logit once, the bitmask, and the per-row words
    it reads (mode, top_k, temperature)."""
    b = np.asarray(inp["x"]).nbytes + 12 * inp["B"]
    if inp.get("bitmask") is not None:
        b += np.asarray(inp["bitmask"]).nbytes
    return b


def merge_alg_bytes(inp, out_bytes_per_row=12):
    """Row merge kernel: per row the candidate set at the method's minimum
    (k (key, index) pairs of 8 B for a stochastic row, one for a greedy row),
    the history and bias lists with one logit gather per listed id, the
    per-request parameters, and the outputs."""
    B = inp["B"]
    esz = 2 if inp["dtype"] == "bf16" else 4
    mode = np.asarray(inp["mode"])
    tk = np.asarray(inp["top_k"])
    temp = np.asarray(inp["temperature"])
    kmax = inp["k_max"]
    cand = 0
    for b in range(B):
        greedy = (mode[b] & 0x040) or ((mode[b] & 0x020) and temp[b] <= 0)
        if greedy:
            cand += 8
        else:
            k = int(tk[b]) if (mode[b] & 0x080) and tk[b] >= 1 else kmax
            cand += 8 * min(k, kmax)
    nh = int(np.asarray(inp["hist_offsets"])[-1]) if inp.get("hist_offsets") is not None else 0
    nb = int(np.asarray(inp["bias_offsets"])[-1]) if inp.get("bias_offsets") is not None else 0
    lists = nh * (4 + esz) + nb * (8 + esz) + 8 * (B + 1)
    return cand + lists + 48 * B + out_bytes_per_row * B


def kernel_source_hash():
    h = hashlib.sha256()
    for p in ("paper_2607_20475_amd/csrc/ss_kernel.hip", "paper_2607_20475_amd/csrc/ss_device.hpp"):
        with open(os.path.join(ROOT, p), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def load_traffic(workload, kernel):
    """HBM bytes per launch of one kernel from the committed rocprofv3 counter
    summary, or None when the kernel source changed since it was taken."""
    p = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(p):
        return None
    with open(p) as f:
        d = json.load(f)
    e = d.get(workload, {}).get(kernel)
    if not e or e.get("kernel_hash") != kernel_source_hash():
        return None
    return e.get("bytes_per_launch")


def traffic_from(fetch_dir, write_dir, out_path, workload):
    """Per-launch HBM bytes of both kernels from two rocprofv3 --pmc runs."""
    import csv
    import glob

    def per_kernel(d, counter):
        f = glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True)
        if not f:
            raise SystemExit(f"no counter_collection.csv under {d}")
        acc = {}
        with open(f[0]) as fh:
            for r in csv.DictReader(fh):
                if r["Counter_Name"] != counter:
                    continue
                n = r["Kernel_Name"]
                key = ("stream" if "ss_stream_kernel" in n else "merge" if "ss_merge_kernel" in n
                       else "copy" if "copyBuffer" in n and int(r["Grid_Size"]) > 0 else None)
                if key is None:
                    continue
                acc.setdefault(key, []).append(float(r["Counter_Value"]) * 1024.0)
        return acc

    fe, wr = per_kernel(fetch_dir, "FETCH_SIZE"), per_kernel(write_dir, "WRITE_SIZE")
    copy_bytes = 16 << 20  # the bench's logit-buffer clones: 64 x 131072 bf16
    # the largest copies are the 16 MiB clones (smaller ones are parameter uploads)
    cf = sorted(fe["copy"])[-1] / copy_bytes
    cw = sorted(wr["copy"])[-1] / copy_bytes
    out = {}
    if os.path.exists(out_path):
        with open(out_path) as fh:
            out = json.load(fh)
    ent = {}
    for k in ("stream", "merge"):
        f = float(np.mean(fe[k])) / cf
        w = float(np.mean(wr[k])) / cw
        ent[k] = dict(bytes_per_launch=f + w, fetch_bytes=f, write_bytes=w, launches=len(fe[k]),
                      kernel_hash=kernel_source_hash())
    ent["copy_scale"] = dict(fetch=cf, write=cw, copy_bytes=copy_bytes)
    out[workload] = ent
    with open(out_path, "w") as fh:
        json.dump(out, fh, indent=1)
    print(json.dumps(out[workload]))


def cpu_baseline(inp, min_seconds, min_reps=4):
    """The oracle on the host: whole batches of the same workload (positions
    varied) until at least `min_seconds` of wall time have passed."""
    import oracle
    nthreads = os.cpu_count() or 1
    omp = os.environ.get("OMP_NUM_THREADS")
    if omp and omp.isdigit():
        nthreads = min(nthreads, int(omp))
    oracle.sample(inp, nthreads=nthreads)  # load + warm
    t0 = time.perf_counter()
    reps = 0
    while reps < min_reps or time.perf_counter() - t0 < min_seconds:
        inp2 = dict(inp)
        inp2["position"] = inp["position"] + reps
        oracle.sample(inp2, nthreads=nthreads)
        reps += 1
    dt = time.perf_counter() - t0
    rows = reps * inp["B"]
    return dict(value=rows / dt, unit="rows/s", cores=nthreads, kind="oracle",
                sample=f"{reps} batches x {inp['B']} rows of the same workload (positions varied), "
                       f"{dt:.2f} s wall on {nthreads} threads")


def bench_sample(args, torch, ssb, W):
    inp = W.config1()
    B, V, kmax = inp["B"], inp["V"], inp["k_max"]
    dev = "cuda"
    x0 = ssb.logits_tensor(inp, dev)
    buf_bytes = x0.numel() * x0.element_size()
    R = max(2, -(-2 * MALL_BYTES // buf_bytes))
    xs = [x0] + [x0.clone() for _ in range(R - 1)]
    prm = ssb.Params.from_arrays(inp, dev)
    ws = ssb.workspace(ssb.OP_SAMPLE, B, V, 0, kmax, ssb.BF16, dev)
    tok = torch.empty(B, dtype=torch.int32, device=dev)
    lp = torch.empty(B, dtype=torch.float32, device=dev)
    fl = torch.empty(B, dtype=torch.int32, device=dev)

    def step(i):
        ssb.sample(xs[i % R], prm, kmax, out_token=tok, out_logprob=lp, flags=fl, ws=ws)

    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()

    # graphs of G steps cycling through the buffers
    G = min(R, args.steps)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        for i in range(G):
            step(i)
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g_full = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g_full):
        for i in range(G):
            step(i)
    rem = args.steps % G
    g_rem = None
    if rem:
        g_rem = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g_rem):
            for i in range(rem):
                step(i)
    n_full = args.steps // G
    for _ in range(2):
        g_full.replay()
    torch.cuda.synchronize()

    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record()
    for _ in range(n_full):
        g_full.replay()
    if g_rem is not None:
        g_rem.replay()
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1)
    ms_per_step = ms / args.steps

    # per-kernel durations: three events per step recorded by the library
    n_k = min(args.steps, 256)
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(n_k)]
    for e3 in evs:
        for e in e3:
            e.record()  # creates the HIP event handles
    torch.cuda.synchronize()
    try:
        for i in range(n_k):
            ssb.set_kernel_events(*evs[i])
            step(i)
    finally:
        ssb.set_kernel_events()
    torch.cuda.synchronize()
    stream_ms = [e[0].elapsed_time(e[1]) for e in evs]
    merge_ms = [e[1].elapsed_time(e[2]) for e in evs]
    kernel_us = {"stream": 1000.0 * float(np.mean(stream_ms)), "merge": 1000.0 * float(np.mean(merge_ms)),
                 "stream_median": 1000.0 * float(np.median(stream_ms)),
                 "merge_median": 1000.0 * float(np.median(merge_ms)), "launches": n_k}
    return inp, ms_per_step, kernel_us, R, fl


def bench_verify(args, torch, ssb, W):
    inp = W.config4()
    B, L, V, kmax = inp["B"], inp["L"], inp["V"], inp["k_max"]
    dev = "cuda"
    x0 = ssb.logits_tensor(inp, dev)
    q = torch.from_numpy(np.ascontiguousarray(inp["draft_probs"])).to(dev)
    d = torch.from_numpy(np.ascontiguousarray(inp["draft_tokens"])).to(dev)
    R = max(2, -(-2 * MALL_BYTES // (x0.numel() * x0.element_size())))
    xs = [x0] + [x0.clone() for _ in range(R - 1)]
    prm = ssb.Params.from_arrays(inp, dev)
    ws = ssb.workspace(ssb.OP_VERIFY, B, V, L, kmax, ssb.BF16, dev)
    out = torch.empty(B, L + 1, dtype=torch.int32, device=dev)
    na = torch.empty(B, dtype=torch.int32, device=dev)
    fl = torch.empty(B, dtype=torch.int32, device=dev)

    def step(i):
        ssb.verify(xs[i % R], q, d, prm, kmax, out_tokens=out, out_nacc=na, flags=fl, ws=ws)

    for i in range(max(4, args.warmup // 4)):
        step(i)
    torch.cuda.synchronize()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        for i in range(R):
            step(i)
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        for i in range(R):
            step(i)
    g.replay()
    torch.cuda.synchronize()
    reps = max(1, args.steps // (4 * R))
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        g.replay()
    e1.record()
    torch.cuda.synchronize()
    us = 1000.0 * e0.elapsed_time(e1) / (reps * R)
    logits = x0.numel() * x0.element_size()
    gathers = B * L * (kmax + 1) * 4  # upper bound of q gathered on the kept sets
    alg = logits + _params_bytes(inp) + d.numel() * 4 + B * (L + 2) * 4 + gathers
    return dict(workload="multistep verification B=64 L=4 V=131072 bf16 target, fp32 draft",
                us_per_batch=us, requests_per_s=B / (us * 1e-6), rows_per_s=B * (L + 1) / (us * 1e-6),
                alg_bytes=alg, GBps=alg / (us * 1e-6) / 1e9, steps=reps * R)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=1024)
    ap.add_argument("--warmup", type=int, default=32)
    ap.add_argument("--no-cpu", action="store_true", help="skip the oracle CPU baseline")
    ap.add_argument("--no-verify", action="store_true", help="skip the secondary verification measurement")
    ap.add_argument("--cpu-seconds", type=float, default=10.0, help="wall time of the oracle baseline sample")
    ap.add_argument("--traffic-from", nargs=3, metavar=("FETCH_DIR", "WRITE_DIR", "OUT"),
                    help="write per-launch HBM bytes from two rocprofv3 --pmc runs, then exit")
    args = ap.parse_args()
    if args.traffic_from:
        traffic_from(*args.traffic_from, workload="cfg1_sample")
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py: this build runs on one GPU only; --gpus must be 1 "
              "(rows are independent, so a multi-GPU run would shard the batch with no communication)",
              file=sys.stderr)
        sys.exit(2)

    import torch
    from gen import workloads as W
    from paper_2607_20475_amd import binding as ssb
    ssb.lib()

    inp, ms_per_step, kernel_us, R, fl = bench_sample(args, torch, ssb, W)
    B = inp["B"]
    logits_b, path_b = algorithmic_bytes(inp)
    us = ms_per_step * 1000.0
    fallback_rows = int(((fl.cpu().numpy() & ssb.FLAG_FALLBACK) > 0).sum())
    names = {"stream": "ss_stream_kernel<bf16>", "merge": "ss_merge_kernel<bf16, sample>"}
    alg = {"stream": stream_alg_bytes(inp), "merge": merge_alg_bytes(inp)}
    kern = {}
    for k in ("stream", "merge"):
        a = alg[k] / (kernel_us[k] * 1e-6) / 1e9
        kern[k] = {"kernel": names[k], "us": kernel_us[k], "us_median": kernel_us[k + "_median"],
                   "alg_bytes_per_launch": alg[k], "achieved": a, "frac": a / HBM_PEAK_GBS,
                   "traffic": load_traffic("cfg1_sample", k)}
    dom = max(("stream", "merge"), key=lambda k: kernel_us[k])
    d = kern[dom]

    res = {
        "metric": METRIC,
        "value": B / (ms_per_step * 1e-3),
        "unit": "rows/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": "heterogeneous singular batch: fused sample B=64 V=131072 bf16, "
                               "mixed greedy/stochastic, penalties, history 512, sparse bias 16",
                   "B": B, "V": inp["V"], "k_max": inp["k_max"], "rotated_buffers": R},
        "us_per_batch": us,
        "path_GBps": path_b / (us * 1e-6) / 1e9,
        "path_frac": path_b / (us * 1e-6) / 1e9 / HBM_PEAK_GBS,
        "path_alg_bytes": path_b,
        "fallback_rows": fallback_rows,
        "roofline": {"bound": "hbm", "kernel": d["kernel"], "achieved": d["achieved"], "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": d["frac"], "traffic": d["traffic"],
                     "alg_bytes_per_launch": d["alg_bytes_per_launch"], "kernel_us": d["us"],
                     "launches_timed": kernel_us["launches"]},
        "kernels": kern,
    }
    if not args.no_verify:
        res["verify"] = bench_verify(args, torch, ssb, W)
    if not args.no_cpu:
        res["cpu_baseline"] = cpu_baseline(inp, args.cpu_seconds)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
