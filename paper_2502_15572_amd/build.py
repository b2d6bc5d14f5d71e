"""Build the HIP retrieval library (gfx950) in-tree: libdresd.so.

The scan file is compiled as six translation units in parallel (one per
scan variant, one for layout/dispatch), beside the merge and the runtime.
Usage: python -m paper_2502_15572_amd.build [-v]
"""
from __future__ import annotations

import concurrent.futures as cf
import hashlib
import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
OUT = os.path.join(HERE, "libdresd.so")
ARCH = os.environ.get("DRESD_OFFLOAD_ARCH", "gfx950")

HIPCC_FLAGS = [
    "--offload-arch=" + ARCH,
    "-O3",
    "-std=c++17",
    "-fPIC",
    # no packed-fp32 instructions in any generated code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-result",
]

# (source, extra defines, object name)
UNITS = [("dresd_kernels.hip", ["-DDRESD_TU=%d" % t], "kernels%d" % t) for t in range(6)] + [
    ("dresd_scan_mq.hip", ["-DDRESD_MQ_TU=0"], "scanmq0"),
    ("dresd_scan_mq.hip", ["-DDRESD_MQ_TU=1"], "scanmq1"),
    ("dresd_merge.hip", [], "merge"), ("dresd_transform.hip", [], "transform"),
    ("dresd_drafts.hip", [], "drafts"), ("dresd_parts.hip", [], "parts"),
    ("dresd_kmeans.hip", [], "kmeans"), ("dresd_bwprobe.hip", [], "bwprobe"),
    ("dresd_runtime.hip", [], "runtime")]


def _compile(hipcc, src, defs, obj, verbose):
    cmd = [hipcc, *HIPCC_FLAGS, *defs, "-I", os.path.join(ROOT, "include"), "-I", CSRC, "-c",
           os.path.join(CSRC, src), "-o", obj]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    err = "\n".join(l for l in r.stderr.splitlines() if "packed-fp32-ops' is not a recognized" not in l)
    if r.returncode != 0:
        raise RuntimeError("hipcc failed for %s:\n%s" % (src, err))
    if err.strip() and verbose:
        print(err, flush=True)
    return obj


def _unit_key(src, defs):
    """Hash of a unit's source, every header it may include, and its flags."""
    h = hashlib.sha256()
    h.update(" ".join(HIPCC_FLAGS + list(defs)).encode())
    for d in (CSRC, os.path.join(ROOT, "include")):
        for f in sorted(os.listdir(d)):
            if f.endswith(".h"):
                h.update(f.encode() + open(os.path.join(d, f), "rb").read())
    h.update(open(os.path.join(CSRC, src), "rb").read())
    return h.hexdigest()[:24]


def build(verbose: bool = False, jobs: int | None = None, cache_dir: str | None = None) -> str:
    """Compile every unit and link libdresd.so.  With cache_dir, objects of
    units whose sources, headers and flags are unchanged are reused."""
    hipcc = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
    tag = "%d" % os.getpid()
    objs = [os.path.join(CSRC, "_%s.%s.o" % (name, tag)) for _, _, name in UNITS]
    jobs = jobs or min(len(UNITS), max(1, (os.cpu_count() or 2)))
    cached = [None] * len(UNITS)
    if cache_dir:
        os.makedirs(cache_dir, exist_ok=True)
        for i, (src, defs, name) in enumerate(UNITS):
            c = os.path.join(cache_dir, "%s.%s.o" % (name, _unit_key(src, defs)))
            cached[i] = c
            if os.path.exists(c):
                objs[i] = c
    try:
        with cf.ThreadPoolExecutor(jobs) as ex:
            futs = [ex.submit(_compile, hipcc, src, defs, obj, verbose)
                    for (src, defs, _), obj in zip(UNITS, objs) if not obj.startswith(cache_dir or "\0")]
            for f in futs:
                f.result()
        for i, c in enumerate(cached):
            if c and objs[i] != c:
                shutil.copyfile(objs[i], c)
        tmp = OUT + ".tmp" + tag
        cmd = [hipcc, "--offload-arch=" + ARCH, "-shared", "-fPIC", *objs, "-o", tmp]
        if verbose:
            print(" ".join(cmd), flush=True)
        subprocess.run(cmd, check=True)
        os.replace(tmp, OUT)
    finally:
        for o in objs:
            if os.path.exists(o) and not (cache_dir and o.startswith(cache_dir)):
                os.remove(o)
    return OUT


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
