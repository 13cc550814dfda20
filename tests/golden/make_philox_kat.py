#!/usr/bin/env python3
"""Regenerate the data rows of philox4x32_10_kat.txt from rocRAND's
Philox4x32-10 (a host build of rocrand/rocrand_philox4x32_10.h; needs
hipcc).  Prints the rows; the fixture's header states their provenance.

    python tests/golden/make_philox_kat.py
"""
import os
import subprocess
import sys
import tempfile

INPUTS = [
    (0x00000000, 0x00000000, 0x00000000, 0x00000000, 0x00000000, 0x00000000),
    (0xFFFFFFFF, 0xFFFFFFFF, 0xFFFFFFFF, 0xFFFFFFFF, 0xFFFFFFFF, 0xFFFFFFFF),
    (0x243F6A88, 0x85A308D3, 0x13198A2E, 0x03707344, 0xA4093822, 0x299F31D0),
]

SRC = r"""
#include <rocrand/rocrand_philox4x32_10.h>
#include <cstdio>
struct K : rocrand_device::philox4x32_10_engine {
  uint4 run(uint4 c, uint2 k) { return ten_rounds(c, k); } };
int main() { K e; unsigned a[6];
  while (scanf("%x %x %x %x %x %x", a, a+1, a+2, a+3, a+4, a+5) == 6) {
    uint4 c = {a[0], a[1], a[2], a[3]}; uint2 k = {a[4], a[5]};
    uint4 r = e.run(c, k); printf("%08x %08x %08x %08x\n", r.x, r.y, r.z, r.w); } }
"""


def main() -> int:
    with tempfile.TemporaryDirectory() as d:
        src = os.path.join(d, "k.cpp")
        with open(src, "w") as f:
            f.write(SRC)
        exe = os.path.join(d, "k")
        subprocess.run(["hipcc", "-x", "hip", "--offload-arch=gfx950", "-O1", src, "-o", exe], check=True)
        inp = "\n".join(" ".join(f"{v:08x}" for v in row) for row in INPUTS) + "\n"
        out = subprocess.run([exe], input=inp, capture_output=True, text=True, check=True).stdout
    for row, line in zip(INPUTS, out.strip().splitlines()):
        print(" ".join(f"{v:08x}" for v in row), line)
    return 0


if __name__ == "__main__":
    sys.exit(main())
