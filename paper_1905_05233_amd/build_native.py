"""Compile the native library ``libwinograd_crt.so`` for gfx950 with hipcc.

Usage: ``python -m paper_1905_05233_amd.build_native [-j JOBS]``.  Objects go
to ``_build/`` at the repository root; the shared library is written next to
this file, where the Python binding loads it.  Always recompiles.
"""
import argparse
import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD = os.path.join(ROOT, "_build")
LIB = os.path.join(PKG, "libwinograd_crt.so")

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"

GEN = os.path.join(BUILD, "gen")   # generated headers (builtin_plans.hpp)
COMMON = ["-O3", "-std=c++17", "-fPIC", "-Wall", f"-I{INCLUDE}", f"-I{CSRC}", f"-I{GEN}"]
# device code: no packed-fp32 instructions (v_pk_*_f32) anywhere
DEVICE = [f"--offload-arch={ARCH}", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
          "-ffp-contract=fast"]

# (source, extra flags, object name)
UNITS = [
    ("rational.cpp", [], "rational.o"),
    ("plan.cpp", [], "plan.o"),
    ("api.hip", DEVICE, "api.o"),
    ("contract.hip", DEVICE, "contract.o"),
    ("transforms.hip", DEVICE + ["-DWG_DTYPE=0"], "transforms_f32.o"),
    ("transforms.hip", DEVICE + ["-DWG_DTYPE=1"], "transforms_f16.o"),
    ("transforms.hip", DEVICE + ["-DWG_DTYPE=2"], "transforms_bf16.o"),
    ("fused.hip", DEVICE + ["-DWG_DTYPE=0"], "fused_f32.o"),
    ("fused.hip", DEVICE + ["-DWG_DTYPE=1"], "fused_f16.o"),
    ("fused.hip", DEVICE + ["-DWG_DTYPE=2"], "fused_bf16.o"),
    ("layer_ops.hip", DEVICE, "layer_ops.o"),
    ("conv1d.hip", DEVICE, "conv1d.o"),
    ("contract_pairwise.hip", DEVICE, "contract_pairwise.o"),
]


def _run(cmd):
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    out = "\n".join(line for line in r.stdout.splitlines() if "packed-fp32-ops" not in line)
    if r.returncode != 0:
        raise RuntimeError(f"command failed ({r.returncode}): {' '.join(cmd)}\n{out}")
    return out


def _newest_header():
    hdrs = [os.path.join(CSRC, f) for f in os.listdir(CSRC) if f.endswith(".hpp")]
    hdrs.append(os.path.join(INCLUDE, "winograd_crt.h"))
    return max(os.path.getmtime(h) for h in hdrs)


def compile_unit(unit, incremental=False):
    src, extra, obj = unit
    path = os.path.join(CSRC, src)
    out = os.path.join(BUILD, obj)
    if incremental and os.path.exists(out):
        if os.path.getmtime(out) > max(os.path.getmtime(path), _newest_header()):
            return ""
    if src.endswith(".cpp"):
        cmd = [HIPCC, "-x", "c++"] + COMMON + ["-c", path, "-o", out]
    else:
        cmd = [HIPCC] + COMMON + extra + ["-c", path, "-o", out]
    return _run(cmd)


def generate_builtin_plans():
    """Build and run the host program that writes builtin_plans.hpp (the fp32
    tables of the built-in plans, from the library's own plan builder)."""
    os.makedirs(GEN, exist_ok=True)
    exe = os.path.join(GEN, "gen_builtin_plans")
    srcs = [os.path.join(CSRC, f) for f in ("gen_builtin_plans.cpp", "plan.cpp", "rational.cpp")]
    _run(["g++", "-O2", "-std=c++17", f"-I{CSRC}", f"-I{INCLUDE}"] + srcs + ["-o", exe])
    _run([exe, os.path.join(GEN, "builtin_plans.hpp")])


def build(jobs=None, verbose=False, incremental=False):
    """Compile every unit (``incremental`` skips objects newer than their
    sources, for development only) and link the shared library."""
    os.makedirs(BUILD, exist_ok=True)
    generate_builtin_plans()
    jobs = jobs or min(8, os.cpu_count() or 4)
    with ThreadPoolExecutor(max_workers=jobs) as ex:
        logs = list(ex.map(lambda u: compile_unit(u, incremental), UNITS))
    objs = [os.path.join(BUILD, u[2]) for u in UNITS]
    tmp = LIB + ".tmp"
    link = [HIPCC, "-shared", "-fPIC", f"--offload-arch={ARCH}"] + objs + ["-o", tmp]
    logs.append(_run(link))
    os.replace(tmp, LIB)
    if verbose:
        for log in logs:
            if log.strip():
                print(log)
    return LIB


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("-j", "--jobs", type=int, default=None)
    ap.add_argument("-v", "--verbose", action="store_true")
    ap.add_argument("--incremental", action="store_true", help="skip up-to-date objects (development)")
    a = ap.parse_args(argv)
    print(build(a.jobs, a.verbose, a.incremental))


if __name__ == "__main__":
    sys.exit(main())
