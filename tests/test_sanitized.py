"""Sanitizer runs on the host code (CPU only).

- The C oracle and a driver program (tests/oracle_asan_driver.c) are built
  together under -fsanitize=address,undefined and run: every oracle call on
  ragged, padded, fp32 and bf16 inputs, each output buffer allocated at
  exactly its contractual size, with no overrun, use after free or leak.
- The C oracle is compiled with -fsanitize=undefined,bounds (trapping,
  static runtime) and its pins are run against that copy: the reference
  arithmetic, indexing and counters stay defined on every pinned input.
- libpair's host code (argument checks, size arithmetic, launch
  preparation) is compiled with the same sanitizer on the host side only
  (device code unchanged), and the host-side ABI tests are run against that
  build: every malformed argument is rejected without undefined behaviour.
Each run happens in a fresh process; a sanitizer report aborts it.
"""
import glob
import os
import subprocess
import sys
import tempfile

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
UBSAN = ["-fsanitize=undefined,bounds", "-fno-sanitize-recover=all"]


def _run(tests, env):
    res = subprocess.run([sys.executable, "-m", "pytest", *tests, "-x", "-q", "-p", "no:cacheprovider",
                          "-m", "not gpu", "-p", "no:xdist"],
                         cwd=ROOT, env=env, capture_output=True, text=True, timeout=900)
    return res.returncode, (res.stdout + res.stderr)[-3000:]


def test_oracle_under_asan():
    with tempfile.TemporaryDirectory() as tmp:
        exe = os.path.join(tmp, "oracle_asan")
        subprocess.run(["gcc", "-O1", "-g", "-std=c11", "-ffp-contract=off", "-fno-fast-math",
                        "-fopenmp", "-fno-omit-frame-pointer", "-fsanitize=address,undefined,bounds",
                        "-fno-sanitize-recover=all", "-o", exe,
                        os.path.join(ROOT, "tests", "oracle_asan_driver.c"),
                        os.path.join(ROOT, "oracle", "pair_oracle.c"), "-lm"],
                       check=True, capture_output=True)
        env = dict(os.environ, OMP_NUM_THREADS="4", ASAN_OPTIONS="detect_leaks=1")
        res = subprocess.run([exe, "200"], env=env, capture_output=True, text=True, timeout=600)
    assert res.returncode == 0, (res.stdout + res.stderr)[-3000:]
    assert "200 cases clean" in res.stdout


def test_oracle_pins_under_ubsan():
    with tempfile.TemporaryDirectory() as tmp:
        so = os.path.join(tmp, "liboracle_ubsan.so")
        subprocess.run(["gcc", "-O1", "-g", "-std=c11", "-ffp-contract=off", "-fno-fast-math",
                        "-fopenmp", "-fPIC", "-shared", *UBSAN, "-static-libubsan", "-o", so,
                        os.path.join(ROOT, "oracle", "pair_oracle.c"), "-lm"],
                       check=True, capture_output=True)
        env = dict(os.environ, PAIR_ORACLE_LIB=so, OMP_NUM_THREADS="4")
        rc, out = _run(["tests/test_oracle_pins.py", "tests/test_oracle_rules.py",
                        "tests/test_oracle_exact.py", "tests/test_oracle_cps.py"], env)
    assert rc == 0, out


def test_host_abi_under_ubsan():
    from paper_2608_11368_amd import build

    rtdirs = glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux")
    if not rtdirs or not glob.glob(os.path.join(rtdirs[0], "libclang_rt.ubsan_standalone-x86_64.so")):
        pytest.skip("no clang UBSan runtime")
    with tempfile.TemporaryDirectory() as tmp:
        so = os.path.join(tmp, "libpair_ubsan.so")
        build.build(out=so, build_dir=os.path.join(tmp, "obj"), host_flags=UBSAN,
                    link_flags=["-fsanitize=undefined", "-shared-libsan",
                                f"-Wl,-rpath,{rtdirs[0]}"])
        env = dict(os.environ, PAIR_LIB=so)
        rc, out = _run(["tests/test_abi.py"], env)
    assert rc == 0, out
