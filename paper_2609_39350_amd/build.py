"""Build libhapmoe.so (HIP, gfx950) in-tree with hipcc."""
import os
import subprocess

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
LIB = os.path.join(PKG, "libhapmoe.so")
SOURCES = ["api.hip", "cost_tables.hip", "stage_dp.hip", "type_dp.hip", "width_dp.hip", "latency_dp.hip", "best_plan.hip"]
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
    "-ffp-contract=off", "-fno-fast-math",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function",
]


CLOCKS_LIB = os.path.join(PKG, "libhapmoe_clocks.so")


def build(force=True, verbose=False, section_clocks=False):
    """Compile every HIP source of the library; returns the .so path.
    section_clocks: the diagnostic variant (libhapmoe_clocks.so) whose stage-DP
    kernel records where its time goes (hapmoe_section_clocks)."""
    lib = CLOCKS_LIB if section_clocks else LIB
    if not force and os.path.exists(lib):
        return lib
    srcs = [os.path.join(PKG, "csrc", s) for s in SOURCES]
    tmp = lib + ".tmp"
    extra = ["-DHAPMOE_SECTION_CLOCKS"] if section_clocks else []
    cmd = [HIPCC, *FLAGS, *extra, "-I", os.path.join(ROOT, "include"), "-I", os.path.join(PKG, "csrc"),
           "-o", tmp, *srcs]
    if verbose:
        print(" ".join(cmd))
    subprocess.run(cmd, check=True)
    os.replace(tmp, lib)
    return lib


if __name__ == "__main__":
    import sys
    print(build(verbose=True, section_clocks="--section-clocks" in sys.argv))
