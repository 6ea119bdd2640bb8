"""Build libdprc.so for gfx950 with hipcc (in-tree, next to this file).

    python -m paper_2605_24879_amd.build [--jobs N] [--debug] [--incremental]

Every .hip source under csrc/ is compiled to an object in _build/ (in
parallel) and linked into paper_2605_24879_amd/libdprc.so.  Packed-fp32 VALU
instructions are disabled for the device code.
"""

import argparse
import concurrent.futures as cf
import os
import re
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
BUILD = os.path.join(HERE, "_build")
LIB = os.path.join(HERE, "libdprc.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"

COMMON = [
    f"--offload-arch={ARCH}", "-std=c++17", "-fPIC", "-Wall", "-Wno-unused-result",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I", os.path.join(ROOT, "include"), "-I", CSRC,
]


def sources():
    return sorted(os.path.join(CSRC, f) for f in os.listdir(CSRC) if f.endswith(".hip"))


def _compile(src, opt):
    obj = os.path.join(BUILD, os.path.basename(src)[:-4] + ".o")
    cmd = [HIPCC, *COMMON, opt, "-c", src, "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    msgs = "\n".join(l for l in (r.stdout + r.stderr).splitlines()
                     if "packed-fp32-ops" not in l and "not a recognized feature" not in l)
    return src, obj, r.returncode, msgs


def _local_includes(path, seen):
    """`path` and the repository headers it includes (quoted #include lines), transitively."""
    if path in seen or not os.path.exists(path):
        return seen
    seen.add(path)
    for line in open(path):
        m = re.match(r'\s*#\s*include\s+"([^"]+)"', line)
        if m:
            _local_includes(os.path.normpath(os.path.join(os.path.dirname(path), m.group(1))), seen)
    return seen


def _stale(src):
    """True when the object of `src` is missing or older than the source or a header it includes."""
    obj = os.path.join(BUILD, os.path.basename(src)[:-4] + ".o")
    if not os.path.exists(obj):
        return True
    return any(os.path.getmtime(d) > os.path.getmtime(obj) for d in _local_includes(src, set()))


def build(jobs=None, debug=False, verbose=False, incremental=False):
    """Compile every source (or, with `incremental`, only those whose object is out of date)
    and link libdprc.so."""
    os.makedirs(BUILD, exist_ok=True)
    opt = "-O1" if debug else "-O3"
    srcs = sources()
    todo = [s for s in srcs if _stale(s)] if incremental else srcs
    objs = [os.path.join(BUILD, os.path.basename(s)[:-4] + ".o") for s in srcs if s not in todo]
    with cf.ThreadPoolExecutor(max_workers=jobs or min(8, max(1, len(todo)))) as ex:
        for src, obj, rc, msgs in ex.map(lambda s: _compile(s, opt), todo):
            if msgs.strip() and (rc != 0 or verbose):
                print(msgs, file=sys.stderr)
            if rc != 0:
                raise RuntimeError(f"hipcc failed on {os.path.basename(src)}")
            objs.append(obj)
    tmp = LIB + ".tmp"
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        print(r.stdout + r.stderr, file=sys.stderr)
        raise RuntimeError("link of libdprc.so failed")
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    ap = argparse.ArgumentParser()
    ap.add_argument("--jobs", type=int, default=None)
    ap.add_argument("--debug", action="store_true")
    ap.add_argument("-v", "--verbose", action="store_true")
    ap.add_argument("--incremental", action="store_true", help="recompile only out-of-date objects")
    a = ap.parse_args()
    print(build(a.jobs, a.debug, a.verbose, a.incremental))
