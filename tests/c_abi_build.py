"""Build tests/c_abi_round (the C ABI used from C++ without Python) against
the in-tree libedit_outer.so.  Called by __graft_entry__.build(); host code
only, linked with a relative rpath so it runs from any checkout."""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
SOURCE = os.path.join(HERE, "c_abi_round.cpp")
PROGRAM = os.path.join(HERE, "c_abi_round")


def build_c_abi_program(hipcc: str = "hipcc") -> str:
    pkg = os.path.join(ROOT, "paper_2412_07210_amd")
    cmd = [hipcc, "--offload-arch=gfx950", "-O2", "-std=c++17", "-Wall",
           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
           "-I", os.path.join(ROOT, "include"), SOURCE, "-o", PROGRAM + ".tmp",
           "-L", pkg, "-l:libedit_outer.so", "-Wl,-rpath,$ORIGIN/../paper_2412_07210_amd"]
    subprocess.run(cmd, check=True, capture_output=True)
    os.replace(PROGRAM + ".tmp", PROGRAM)
    return PROGRAM
