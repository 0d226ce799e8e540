"""Build the CPU emulation library (host-only hipcc, C++20) for the tests."""

import os
import shutil
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
OUT = os.path.join(HERE, "_build", "libacdc_emu.so")
SRC = os.path.join(HERE, "acdc_emu.cpp")
DEPS = [SRC] + [os.path.join(HERE, "..", "..", "paper_1511_05946_amd", "csrc", f)
                for f in os.listdir(os.path.join(HERE, "..", "..", "paper_1511_05946_amd", "csrc"))
                if f.endswith(".hpp")]


def build() -> str:
    if os.path.exists(OUT) and all(os.path.getmtime(OUT) >= os.path.getmtime(d) for d in DEPS):
        return OUT
    hipcc = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    os.makedirs(os.path.dirname(OUT), exist_ok=True)
    tmp = OUT + ".tmp"
    # every plan from 1024 up may run as persistent accumulating workgroups
    # here (acdc_emu_set_backward_slots), not only those that do on the GPU
    subprocess.run([hipcc, "-std=c++20", "-x", "hip", "--offload-host-only", "-O1", "-fPIC", "-shared",
                    "-DACDC_BWD_ACC_MAX_ROWS=16", SRC, "-o", tmp, "-lpthread"], check=True, capture_output=True)
    os.replace(tmp, OUT)
    return OUT


if __name__ == "__main__":
    print(build())
