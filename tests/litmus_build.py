"""Build step of the hand-off litmus program (tests/handoff_litmus.hip) into tests/_build/, run by
__graft_entry__.build() beside the library so that GPU runs only execute it."""
import os
import shutil
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
EXE = os.path.join(HERE, "_build", "handoff_litmus")


def build() -> str:
    hipcc = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    os.makedirs(os.path.dirname(EXE), exist_ok=True)
    cmd = [hipcc, "-O3", "-std=c++17", "--offload-arch=gfx950", "-Xclang", "-target-feature", "-Xclang",
           "-packed-fp32-ops", "-I" + os.path.join(ROOT, "paper_2511_09844_amd", "csrc"),
           "-I" + os.path.join(ROOT, "include"), os.path.join(HERE, "handoff_litmus.hip"), "-o", EXE + ".tmp"]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError("hipcc failed on handoff_litmus.hip:\n" + res.stderr)
    os.replace(EXE + ".tmp", EXE)
    return EXE
