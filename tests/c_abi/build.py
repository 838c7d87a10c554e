"""Builds the standalone C-ABI test program (tests/c_abi/roundtrip) against the
in-tree libmori.so and the C oracle; host code only."""
from __future__ import annotations

import os
import subprocess
import tempfile

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
BIN = os.path.join(HERE, "roundtrip")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")


def build() -> str:
    lib_dir = os.path.join(ROOT, "paper_2606_00866_amd")
    if not os.path.exists(os.path.join(lib_dir, "libmori.so")):
        raise RuntimeError("libmori.so is not built")
    with tempfile.TemporaryDirectory() as tmp:
        obj = os.path.join(tmp, "mori_oracle.o")
        main = os.path.join(tmp, "roundtrip.o")
        steps = [
            ["gcc", "-O2", "-std=c11", "-fPIC", "-c", os.path.join(ROOT, "oracle", "mori_oracle.c"), "-o", obj],
            [HIPCC, "--offload-arch=gfx950", "-O2", "-std=c++17", "-Xclang", "-target-feature", "-Xclang",
             "-packed-fp32-ops", "-I", os.path.join(ROOT, "include"), "-I", os.path.join(ROOT, "oracle"),
             "-c", os.path.join(HERE, "roundtrip.cpp"), "-o", main],
            [HIPCC, "--offload-arch=gfx950", main, obj, "-L", lib_dir, "-lmori",
             "-Wl,-rpath,$ORIGIN/../../paper_2606_00866_amd", "-o", BIN + ".tmp"],
        ]
        for cmd in steps:
            res = subprocess.run(cmd, capture_output=True, text=True)
            if res.returncode != 0:
                raise RuntimeError(f"{cmd[0]} failed:\n{res.stdout}{res.stderr}")
    os.replace(BIN + ".tmp", BIN)
    return BIN


if __name__ == "__main__":
    print(build())
