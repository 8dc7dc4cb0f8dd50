"""CPU sanitizer builds (AddressSanitizer + UndefinedBehaviorSanitizer, no recovery) of the oracle and
of the library's host code, run on the parity-check matrices of the five workloads and two odd-sized
random ones.

- The oracle (C) with a driver that decodes in both modes, with taps, the fp64 word decode forced
  to the canonical codes, per-word alpha, CASA, and the building blocks.
- The library's host code (every source compiled host-only: validation, Tanner lists, the fused
  tile search, weight packing, workspace plans and chunking, launch sequences, the AAP import, the
  spectrum, the training step's host side) linked against a host stand-in for the HIP runtime
  (device memory in host memory, launches that do nothing), with a driver over every entry point.
"""
import os
import re
import subprocess

import numpy as np
import pytest

from workloads import CONFIGS
from workloads.configs import parity_check

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SAN = os.path.join(ROOT, "tests", "sanitize")
CSRC = os.path.join(ROOT, "paper_2410_05911_amd", "csrc")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
SAN_FLAGS = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer"]
ENV = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0", UBSAN_OPTIONS="print_stacktrace=1")


def _codes(tmp_path):
    files = []
    mats = [parity_check(CONFIGS[c]) for c in (1, 2, 3, 4, 5)]
    rng = np.random.default_rng(3)
    for m, n in ((13, 30), (21, 47)):                  # odd sizes: partial tiles, straddling types
        H = np.zeros((m, n), np.uint8)
        for i in range(n):
            H[rng.choice(m, 3, replace=False), i] = 1
        for j in range(m):
            if not H[j].any():
                H[j, rng.integers(n)] = 1
        mats.append(H)
    for k, H in enumerate(mats):
        p = tmp_path / f"H{k}.bin"
        with open(p, "wb") as f:
            f.write(np.array(H.shape, np.int32).tobytes())
            f.write(np.ascontiguousarray(H, np.uint8).tobytes())
        files.append(str(p))
    return files


def _run(cmd, **kw):
    r = subprocess.run(cmd, capture_output=True, text=True, env=ENV, **kw)
    return r.returncode, r.stdout, r.stderr


def test_oracle_under_sanitizers(tmp_path):
    exe = str(tmp_path / "oracle_driver")
    subprocess.run(["gcc", "-std=c11", "-O1", "-g", "-ffp-contract=off", *SAN_FLAGS, "-I", os.path.join(ROOT, "oracle"),
                    os.path.join(ROOT, "oracle", "aecct_oracle.c"), os.path.join(SAN, "oracle_driver.c"), "-lm",
                    "-o", exe], check=True)
    rc, out, err = _run([exe] + _codes(tmp_path), timeout=900)
    assert rc == 0 and "oracle driver ok" in out, (out[-2000:], err[-4000:])
    assert "runtime error" not in err and "AddressSanitizer" not in err, err[-4000:]


def test_library_host_code_under_sanitizers(tmp_path):
    objs = []
    for src in sorted(os.listdir(CSRC)):
        if not src.endswith((".cpp", ".hip")):
            continue
        obj = str(tmp_path / (os.path.splitext(src)[0] + ".o"))
        subprocess.run([HIPCC, "-x", "hip", "--cuda-host-only", "-O1", "-g", "-std=c++17", "-fPIC", "-ffp-contract=off",
                        "-I", os.path.join(ROOT, "include"), "-Xarch_host", SAN_FLAGS[0], "-Xarch_host", SAN_FLAGS[1],
                        "-Xarch_host", SAN_FLAGS[2], "-c", os.path.join(CSRC, src), "-o", obj],
                       check=True, capture_output=True)
        objs.append(obj)
    # the compiler's references to each source's device image: defined empty, never read
    nm = subprocess.run(["nm", "-u", *objs], check=True, capture_output=True, text=True).stdout
    fatbins = sorted(set(re.findall(r"\b(__hip_fatbin_[0-9a-f]+)\b", nm)))
    stub2 = tmp_path / "fatbin_names.cpp"
    stub2.write_text("".join(f'extern "C" const char {f}[16] = {{0}};\n' for f in fatbins))
    clang = "/opt/rocm/llvm/bin/clang++"
    common = ["-O1", "-g", "-std=c++17", "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include", "-I", os.path.join(ROOT, "include"),
              *SAN_FLAGS]
    exe = str(tmp_path / "host_driver")
    subprocess.run([clang, *common, os.path.join(SAN, "host_driver.cpp"), os.path.join(SAN, "hip_host_stub.cpp"),
                    str(stub2), *objs, "-o", exe], check=True)
    rc, out, err = _run([exe] + _codes(tmp_path), timeout=900)
    assert rc == 0 and "host driver ok" in out, (out[-2000:], err[-4000:])
    assert "runtime error" not in err and "AddressSanitizer" not in err, err[-4000:]
