"""The C oracle is free of memory errors and undefined behaviour on the inputs
the pins feed it: fkv_oracle.c is compiled on the CPU with AddressSanitizer
and UndefinedBehaviorSanitizer (gcc, a temporary library), and the whole pin
suite runs against that build in a child pytest process (FKV_ORACLE_LIB), with
the sanitizer runtime preloaded into the Python interpreter.  Any report
aborts the child, which fails this test."""
import os
import shutil
import subprocess
import sys

import pytest

import oracle

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)


def _runtime(name):
    p = subprocess.run(["gcc", f"-print-file-name={name}"], capture_output=True, text=True).stdout.strip()
    return p if os.path.isabs(p) and os.path.exists(p) else None


@pytest.mark.skipif(shutil.which("gcc") is None, reason="needs gcc")
def test_pins_pass_under_asan_and_ubsan(tmp_path):
    asan = _runtime("libasan.so")
    if asan is None:
        pytest.skip("gcc has no AddressSanitizer runtime here")
    src_dir = os.path.dirname(oracle._SRC)
    for f in ("fkv_oracle.c", "fkv_oracle.h"):
        shutil.copy(os.path.join(src_dir, f), tmp_path / f)
    so = tmp_path / "liboracle_san.so"
    flags = ["-O1", "-g", "-std=c11", "-fopenmp", "-fPIC", "-shared", "-ffp-contract=off",
             "-fno-omit-frame-pointer", "-fsanitize=address,undefined", "-fno-sanitize-recover=all"]
    subprocess.run(["gcc", *flags, str(tmp_path / "fkv_oracle.c"), "-o", str(so), "-lm"],
                   check=True, capture_output=True)
    env = dict(os.environ, FKV_ORACLE_LIB=str(so), OMP_NUM_THREADS="4", LD_PRELOAD=asan,
               ASAN_OPTIONS="detect_leaks=0:abort_on_error=1:verify_asan_link_order=0",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                        os.path.join(HERE, "test_oracle_pins.py"), os.path.join(HERE, "test_oracle_profiling_pins.py"),
                        os.path.join(HERE, "test_golden.py")],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=900)
    tail = (r.stdout[-3000:] + "\n" + r.stderr[-3000:])
    assert r.returncode == 0, f"pin suite under the sanitizers failed:\n{tail}"
    assert "ERROR: AddressSanitizer" not in r.stderr and "runtime error:" not in r.stderr, tail
