"""Build libfcm.so (HIP kernels for gfx950 + host planner/C ABI) in-tree.

    python -m paper_2404_19331_amd.build [--jobs N] [--verbose]

Every source under csrc/ is compiled with hipcc into _build/, then linked into
paper_2404_19331_amd/libfcm.so. Sources compile in parallel.
"""
import argparse
import concurrent.futures as cf
import os
import subprocess
import sys
import time

PKG = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(PKG, "csrc")
BUILD = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "libfcm.so")
INCLUDE = os.path.join(os.path.dirname(PKG), "include")

ARCH = "gfx950"
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
COMMON = ["-O3", "-std=c++17", "-fPIC", "-I" + CSRC, "-I" + INCLUDE, "-Wall", "-Wno-unused-function"]
# Packed fp32 VALU instructions stay off: ordinary float code is enough here.
DEVICE = ["--offload-arch=" + ARCH, "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
          # matrix-core accumulators in ordinary VGPRs: no AGPR copies around each MFMA
          "-mllvm", "-amdgpu-mfma-vgpr-form"]


def sources():
    out = []
    for f in sorted(os.listdir(CSRC)):
        if f.endswith(".hip") or f.endswith(".cpp"):
            out.append(os.path.join(CSRC, f))
    return out


def _compile(src, verbose):
    obj = os.path.join(BUILD, os.path.basename(src) + ".o")
    cmd = [HIPCC] + COMMON
    if src.endswith(".hip"):
        cmd += DEVICE
    else:
        cmd += ["-D__HIP_PLATFORM_AMD__"]
    cmd += ["-c", src, "-o", obj]
    t0 = time.time()
    r = subprocess.run(cmd, capture_output=True, text=True)
    msg = "\n".join(l for l in (r.stdout + r.stderr).splitlines()
                    if "not a recognized feature" not in l and l.strip())
    if r.returncode != 0:
        raise RuntimeError("compile failed: %s\n%s\n%s" % (os.path.basename(src), " ".join(cmd), msg))
    if verbose and msg:
        print(msg)
    return obj, time.time() - t0


def build(jobs=None, verbose=False):
    """Compile every source and link libfcm.so. Always rebuilds."""
    os.makedirs(BUILD, exist_ok=True)
    srcs = sources()
    jobs = jobs or min(len(srcs), max(1, min(16, os.cpu_count() or 1)))
    objs = []
    with cf.ThreadPoolExecutor(max_workers=jobs) as ex:
        futs = {ex.submit(_compile, s, verbose): s for s in srcs}
        for f in cf.as_completed(futs):
            obj, dt = f.result()
            objs.append(obj)
            if verbose:
                print("  %-24s %.1fs" % (os.path.basename(futs[f]), dt))
    tmp = LIB + ".tmp%d" % os.getpid()
    cmd = [HIPCC, "--offload-arch=" + ARCH, "-shared", "-fPIC", "-o", tmp] + sorted(objs)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("link failed:\n%s\n%s" % (" ".join(cmd), r.stderr))
    os.replace(tmp, LIB)
    return LIB


def main(argv=None):
    ap = argparse.ArgumentParser()
    ap.add_argument("--jobs", type=int, default=None)
    ap.add_argument("--verbose", action="store_true")
    a = ap.parse_args(argv)
    t0 = time.time()
    path = build(a.jobs, a.verbose)
    print("built %s in %.1fs" % (path, time.time() - t0))


if __name__ == "__main__":
    sys.exit(main())
