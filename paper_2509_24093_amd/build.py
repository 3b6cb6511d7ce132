"""Build ``libcgconv.so`` for gfx950, in-tree.

Steps: compile and run the CG code generator (host C++) into ``_build/``,
compile every translation unit with hipcc for gfx950 in parallel (one unit
per generated L_max), link the shared library next to this file.

    python -m paper_2509_24093_amd.build
"""

from __future__ import annotations

import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
BUILD = os.path.join(HERE, "_build")
LIB = os.path.join(HERE, "libcgconv.so")
PROBE_LIB = os.path.join(HERE, "libhbmprobe.so")  # the benchmark's HBM-ceiling kernels
INCLUDE = os.path.join(os.path.dirname(HERE), "include")
LGEN = 8  # highest L_max with a generated register-resident contraction
FUSED_LMAX = 6  # highest L_max with a fused (second pass + CG + inverse first pass) kernel
MIX_LMAX = 6  # highest L_max with a channel-mixing (MFMA) CG stage
INTER_LMAX = 6  # highest L_max with an inter-channel (MFMA reduction) CG stage
SMALL_LMAX = 6  # highest L_max with the one-block kernel for DFT lengths <= 256
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
# Packed FP32 instructions are disabled for all device code.
HIP_FLAGS = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC",
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
             "-I" + BUILD, "-I" + CSRC, "-I" + INCLUDE]


def _run(cmd, verbose):
    if verbose:
        print("+ " + " ".join(cmd), flush=True)
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    if r.returncode != 0:
        raise RuntimeError("build step failed (%d): %s\n%s" % (r.returncode, " ".join(cmd), r.stdout))
    out = r.stdout.strip()
    if verbose and out:
        # hipcc's host pass warns that it does not know the packed-fp32 feature
        lines = [l for l in out.splitlines() if "packed-fp32-ops" not in l]
        if lines:
            print("\n".join(lines), flush=True)
    return r.stdout


def build(jobs: int | None = None, verbose: bool = True) -> str:
    os.makedirs(BUILD, exist_ok=True)
    gen = os.path.join(BUILD, "gen_cg")
    _run(["g++", "-O2", "-std=c++17", os.path.join(CSRC, "codegen", "gen_cg.cpp"),
          os.path.join(CSRC, "cg_table.cpp"), "-o", gen], verbose)
    _run([gen, BUILD, str(LGEN)], verbose)

    units = [
        (["g++", "-O2", "-std=c++17", "-fPIC", "-c"], "cg_table.cpp", "cg_table.o", []),
        ([HIPCC, "-x", "hip", "-c"] + HIP_FLAGS, "cgconv.cpp", "cgconv.o", []),
        ([HIPCC, "-c"] + HIP_FLAGS, "fft.hip", "fft.o", []),
        ([HIPCC, "-c"] + HIP_FLAGS, "cg.hip", "cg.o", []),
        ([HIPCC, "-c"] + HIP_FLAGS, "gft.hip", "gft.o", []),
    ]
    for L in range(LGEN, -1, -1):  # largest first: it compiles longest
        units.append(([HIPCC, "-c"] + HIP_FLAGS, "cg_gen.hip", "cg_gen_L%d.o" % L,
                      ["-DCGCONV_TU_L=%d" % L, '-DCGCONV_BODY="cg_body_L%d.inc"' % L]))
    for L in range(FUSED_LMAX, -1, -1):
        units.append(([HIPCC, "-c"] + HIP_FLAGS, "cg_fused.hip", "cg_fused_L%d.o" % L,
                      ["-DCGCONV_TU_L=%d" % L, '-DCGCONV_BODY="cg_body_L%d.inc"' % L]))
    for L in range(MIX_LMAX, -1, -1):
        units.append(([HIPCC, "-c"] + HIP_FLAGS, "cg_mix.hip", "cg_mix_L%d.o" % L,
                      ["-DCGCONV_TU_L=%d" % L, '-DCGCONV_BODY="cg_body_L%d.inc"' % L]))
    for L in range(INTER_LMAX, -1, -1):
        units.append(([HIPCC, "-c"] + HIP_FLAGS, "cg_inter.hip", "cg_inter_L%d.o" % L,
                      ["-DCGCONV_TU_L=%d" % L, '-DCGCONV_BODY="cg_body_L%d.inc"' % L]))
    for L in range(SMALL_LMAX, -1, -1):
        units.append(([HIPCC, "-c"] + HIP_FLAGS, "cg_small.hip", "cg_small_L%d.o" % L,
                      ["-DCGCONV_TU_L=%d" % L, '-DCGCONV_BODY="cg_body_L%d.inc"' % L]))
    for L in range(LGEN, -1, -1):
        units.append(([HIPCC, "-c"] + HIP_FLAGS, "gate.hip", "gate_L%d.o" % L,
                      ["-DCGCONV_TU_L=%d" % L, '-DCGCONV_BODY="cg_body_L%d.inc"' % L]))
    objs = []

    def compile_unit(u):
        base, src, obj, extra = u
        o = os.path.join(BUILD, obj)
        _run(base + extra + [os.path.join(CSRC, src), "-o", o], verbose)
        return o

    n = jobs or min(8, os.cpu_count() or 4)
    with ThreadPoolExecutor(max_workers=n) as ex:
        objs = list(ex.map(compile_unit, units))
    tmp = LIB + ".tmp"
    _run([HIPCC, "-shared", "-fPIC", "--offload-arch=gfx950", "-o", tmp] + objs, verbose)
    os.replace(tmp, LIB)
    tmp = PROBE_LIB + ".tmp"
    _run([HIPCC, "-shared"] + HIP_FLAGS + [os.path.join(CSRC, "hbm_probe.hip"), "-o", tmp], verbose)
    os.replace(tmp, PROBE_LIB)
    return LIB


if __name__ == "__main__":
    build(verbose="-q" not in sys.argv)
    print("built", LIB)
