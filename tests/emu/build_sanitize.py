"""Build the sanitizer driver (tests/emu/sanitize_driver.cpp): the CPU
emulation and the library's host code, compiled for the host only with
AddressSanitizer and UndefinedBehaviorSanitizer.  Test infrastructure; no
GPU code is built here."""

import os
import shutil
import subprocess
import tempfile

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
CSRC = os.path.join(ROOT, "paper_1511_05946_amd", "csrc")
OUT = os.path.join(HERE, "_build", "sanitize_driver")
SRCS = [os.path.join(HERE, "sanitize_driver.cpp"), os.path.join(CSRC, "acdc_api.hip"),
        os.path.join(CSRC, "acdc_multipass.hip")]
SAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
       "-Xarch_host", "-fno-sanitize-recover=all", "-Xarch_host", "-fno-omit-frame-pointer"]
# -O0 keeps the sanitized build of the template-heavy sources under a minute;
# ACDC_PLAN_SUBSET instantiates a few widths of each kind, the same set in
# every object.  The .hip sources are compiled with their device code (never
# launched here) so that they link; only host code is sanitized.
COMMON = ["-std=c++20", "-O0", "-gline-tables-only", "-DACDC_PLAN_SUBSET",
          "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops", "-Wno-unused-command-line-argument"]


def deps():
    out = list(SRCS) + [os.path.join(HERE, "acdc_emu.cpp"), os.path.join(ROOT, "include", "acdc.h")]
    out += [os.path.join(CSRC, f) for f in os.listdir(CSRC) if f.endswith(".hpp")]
    return out


def build() -> str:
    if os.path.exists(OUT) and all(os.path.getmtime(OUT) >= os.path.getmtime(d) for d in deps()):
        return OUT
    hipcc = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    os.makedirs(os.path.dirname(OUT), exist_ok=True)
    with tempfile.TemporaryDirectory(prefix="acdc_san_") as tmp:
        objs, procs = [], []
        for src in SRCS:
            obj = os.path.join(tmp, os.path.basename(src) + ".o")
            kind = ["-x", "hip", "--offload-host-only"] if src.endswith(".cpp") else ["--offload-arch=gfx950"]
            cmd = [hipcc, *COMMON, *kind, *SAN, "-I", os.path.join(ROOT, "include"), "-I", CSRC, "-c", src,
                   "-o", obj]
            procs.append(subprocess.Popen(cmd, stdout=subprocess.PIPE, stderr=subprocess.PIPE, text=True))
            objs.append(obj)
        for proc in procs:
            out, err = proc.communicate()
            if proc.returncode != 0:
                raise RuntimeError(f"sanitizer build failed:\n{out}{err}")
        tmp_out = OUT + ".tmp"
        cmd = [hipcc, "--offload-arch=gfx950", *SAN, *objs, "-o", tmp_out, "-lpthread"]
        proc = subprocess.run(cmd, capture_output=True, text=True)
        if proc.returncode != 0:
            raise RuntimeError(f"sanitizer link failed:\n{proc.stdout}{proc.stderr}")
        os.replace(tmp_out, OUT)
    return OUT


if __name__ == "__main__":
    print(build())
