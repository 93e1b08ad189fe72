"""Compile the HIP kernels and the C ABI into ``lib/librandattn.so`` (gfx950).

Run as ``python -m paper_2609_03430_amd.build``; ``__graft_entry__.build()``
calls :func:`build`.  Every source is compiled on every call.
"""

import concurrent.futures
import json
import os
import re
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
LIBDIR = os.path.join(PKG, "lib")
LIB = os.path.join(LIBDIR, "librandattn.so")
OBJDIR = os.path.join(ROOT, "_build")
# per-kernel register, scratch and LDS use reported by the compiler
RESOURCES = os.path.join(OBJDIR, "kernel_resources.json")
SOURCES = ["attention.hip", "evict.hip", "state.hip", "window_score.hip", "scored.hip", "api.cpp"]

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC",
    "-I" + os.path.join(ROOT, "include"), "-I" + CSRC,
    # packed fp32 VALU forms stay off in all device code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function",
    "-Rpass-analysis=kernel-resource-usage",
]


def parse_resources(stderr):
    """{kernel: {field: value}} from the compiler's resource-usage remarks."""
    out, cur = {}, None
    for line in stderr.splitlines():
        m = re.search(r"remark: Function Name: (\S+)", line)
        if m:
            cur = out.setdefault(m.group(1), {})
            continue
        m = re.search(r"remark:\s+([A-Za-z][A-Za-z /\[\]]*?): (\S+) \[-Rpass-analysis", line)
        if m and cur is not None:
            val = m.group(2)
            cur[m.group(1)] = int(val) if val.isdigit() else val
    return out


def _compile(src):
    obj = os.path.join(OBJDIR, os.path.basename(src) + ".o")
    cmd = [HIPCC] + FLAGS + ["-x", "hip", "-c", os.path.join(CSRC, src), "-o", obj]
    res = subprocess.run(cmd, capture_output=True, text=True)
    noise = "is not a recognized feature for this target"
    kept = []
    for l in res.stderr.splitlines():
        if noise in l or "kernel-resource-usage" in l:
            continue
        if l.lstrip().startswith(("|", "^")) or re.match(r"\s+\d+ \|", l):
            continue                      # source excerpts of the remarks
        kept.append(l)
    err = "\n".join(kept)
    if res.returncode != 0:
        raise RuntimeError("compile failed: %s\n%s" % (" ".join(cmd), err))
    return obj, err, parse_resources(res.stderr)


def build(verbose=False):
    """Compile every source and link the shared library; returns its path."""
    os.makedirs(OBJDIR, exist_ok=True)
    os.makedirs(LIBDIR, exist_ok=True)
    with concurrent.futures.ThreadPoolExecutor(len(SOURCES)) as ex:
        results = list(ex.map(_compile, SOURCES))
    if verbose:
        for obj, err, _ in results:
            if err.strip():
                print(err, file=sys.stderr)
    resources = {}
    for src, (_, _, r) in zip(SOURCES, results):
        for name, fields in r.items():
            resources[name] = dict(fields, source=src)
    with open(RESOURCES, "w") as f:
        json.dump(resources, f, indent=0, sort_keys=True)
    tmp = LIB + ".tmp"
    cmd = [HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp] + \
        [obj for obj, _, _ in results]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError("link failed: %s\n%s" % (" ".join(cmd), res.stderr))
    shutil.move(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
