"""pytest plugin for test_abi_sanitized.py: the binding loads the library
build named by FKV_SANITIZED_LIB (host code built with AddressSanitizer and
UndefinedBehaviorSanitizer) instead of the package's libfkv.so, and the run
fails unless that build is the one mapped into the process."""
import os

import paper_2605_09681_amd as fkv

fkv.LIB_PATH = os.environ["FKV_SANITIZED_LIB"]


def pytest_sessionfinish(session, exitstatus):
    with open("/proc/self/maps") as f:
        mapped = any(fkv.LIB_PATH in line for line in f)
    if not mapped:
        session.exitstatus = 1
        print(f"\nsanitized library {fkv.LIB_PATH} was not loaded")
