"""Builds libss.so (gfx950) from the HIP sources in csrc/ with hipcc.

Every kernel instantiation sits in a translation unit of its own (the merge
source is compiled once per (element type, operation) pair), and the units
compile in parallel before one link step.
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
OBJ_DIR = os.path.join(HERE, "_build")
LIB_PATH = os.path.join(HERE, "libss.so")
# measurement aid of bench.py (a plain streaming read), kept out of libss.so
BENCH_LIB_PATH = os.path.join(HERE, "libss_bench.so")
HEADERS = [os.path.join(CSRC, h) for h in ("ss_impl.hpp", "ss_device.hpp", "ss_launch.hpp")] + [
    os.path.join(ROOT, "include", "ss.h")
]

HIPCC_FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC",
    # exact float32 prologue: no contraction, correctly rounded division
    "-ffp-contract=off", "-fhip-fp32-correctly-rounded-divide-sqrt",
    # no packed-FP32 instructions
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I" + os.path.join(ROOT, "include"),
]

_DT = {"f32": 0, "bf16": 1}
_OP = {"topk": 0, "sample": 1, "verify": 2, "process": 3, "logprobs": 4, "sample_x": 5}


def units() -> list[tuple[str, str, list[str]]]:
    """(object name, source, extra flags) of every translation unit."""
    u = [
        ("ss_api", "ss_api.hip", []),
        ("ss_stream", "ss_stream.hip", []),
        ("ss_aux", "ss_aux.hip", []),
        ("ss_noalloc", "ss_noalloc.hip", []),
    ]
    for dn, dv in _DT.items():
        for on, ov in _OP.items():
            u.append(("ss_merge_%s_%s" % (dn, on), "ss_merge.hip",
                      ["-DSS_MERGE_DT=%d" % dv, "-DSS_MERGE_OP=%d" % ov]))
    return [x for x in u if os.path.exists(os.path.join(CSRC, x[1]))]


def _compile(hipcc: str, name: str, src: str, extra: list[str], incremental: bool) -> str:
    obj = os.path.join(OBJ_DIR, name + ".o")
    srcp = os.path.join(CSRC, src)
    if incremental and os.path.exists(obj):
        t = os.path.getmtime(obj)
        if all(os.path.getmtime(d) <= t for d in [srcp] + HEADERS):
            return obj
    tmp = obj + ".tmp%d" % os.getpid()
    cmd = [hipcc] + HIPCC_FLAGS + extra + ["-c", "-o", tmp, srcp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("hipcc failed on %s:\n%s%s" % (name, r.stdout, r.stderr))
    os.replace(tmp, obj)
    return obj


def build(verbose: bool = False, incremental: bool = False, jobs: int | None = None) -> str:
    hipcc = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
    os.makedirs(OBJ_DIR, exist_ok=True)
    us = units()
    jobs = jobs or min(len(us), max(1, os.cpu_count() or 1))
    with cf.ThreadPoolExecutor(max_workers=jobs) as ex:
        futs = [ex.submit(_compile, hipcc, n, s, e, incremental) for n, s, e in us]
        objs = [f.result() for f in futs]
    tmp = LIB_PATH + ".tmp%d" % os.getpid()
    cmd = [hipcc, "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp] + objs
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("link failed:\n" + r.stdout + r.stderr)
    if verbose and r.stderr:
        print(r.stderr)
    os.replace(tmp, LIB_PATH)
    src = os.path.join(CSRC, "bench_probe.hip")
    if os.path.exists(src):
        tmp = BENCH_LIB_PATH + ".tmp%d" % os.getpid()
        r = subprocess.run([hipcc] + HIPCC_FLAGS + ["-shared", "-o", tmp, src], capture_output=True, text=True)
        if r.returncode != 0:
            raise RuntimeError("hipcc failed on bench_read:\n" + r.stdout + r.stderr)
        os.replace(tmp, BENCH_LIB_PATH)
    return LIB_PATH


def is_stale() -> bool:
    if not os.path.exists(LIB_PATH):
        return True
    t = os.path.getmtime(LIB_PATH)
    deps = HEADERS + [os.path.join(CSRC, s) for _, s, _ in units()]
    deps += [os.path.join(CSRC, "bench_probe.hip")] if os.path.exists(os.path.join(CSRC, "bench_probe.hip")) else []
    return any(os.path.getmtime(d) > t for d in deps)


if __name__ == "__main__":
    print(build(verbose=True, incremental="--incremental" in sys.argv))
