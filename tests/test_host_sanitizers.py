"""Host code under AddressSanitizer + UndefinedBehaviorSanitizer (CPU only).

The segment-table validation, plan packing and argument checks of the library
(plan.cpp, api.cpp) are integer indexing over caller-supplied tables.  This
test builds the host-sanitized variant of the library (those two files under
g++ -fsanitize=address,undefined; the device code as usual) and a sanitized
build of the oracle, then runs the host-side test files against them in a
child process with gcc's libasan loaded first:

* tests/test_plan.py -- packing against the independent packer, random valid
  and defective tables, every validation error, the argument checks of every
  entry point, workspace queries;
* tests/test_oracle.py -- the oracle's pins.

A sanitizer report ends the child with a failure (UBSan is built without
recovery, ASan always aborts), and the child first checks that the sanitized
libraries are the ones mapped.
"""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

_CHECK_LOADED = r"""
import os, sys
from paper_2607_28848_amd import dsv
import oracle
oracle.threads()
maps = open("/proc/self/maps").read()
need = [os.environ["DSV_LIBRARY"], os.environ["DSVO_LIBRARY"], "libasan.so"]
missing = [n for n in need if n not in maps]
assert dsv.LIB_PATH == os.environ["DSV_LIBRARY"], dsv.LIB_PATH
assert not missing, missing
print("sanitized libraries mapped")
"""


def _gcc_runtime(name):
    out = subprocess.run(["gcc", "-print-file-name=" + name], capture_output=True, text=True).stdout.strip()
    return out if os.path.isabs(out) and os.path.exists(out) else None


def test_host_code_clean_under_asan_and_ubsan():
    asan, ubsan = _gcc_runtime("libasan.so"), _gcc_runtime("libubsan.so")
    if not (asan and ubsan):
        pytest.skip("gcc's sanitizer runtimes are not installed")
    sys.path.insert(0, ROOT)
    from paper_2607_28848_amd import build as pkg_build
    import oracle
    dsv_lib = pkg_build.build_host_asan()
    dsvo_lib = oracle.build_asan()
    env = dict(os.environ)
    pre = env.get("LD_PRELOAD")
    env.update({
        "LD_PRELOAD": asan + ":" + ubsan + ((":" + pre) if pre else ""),
        "ASAN_OPTIONS": "detect_leaks=0:verify_asan_link_order=0:abort_on_error=1",
        "UBSAN_OPTIONS": "print_stacktrace=1:halt_on_error=1",
        "DSV_LIBRARY": dsv_lib,
        "DSVO_LIBRARY": dsvo_lib,
        "PYTHONPATH": ROOT + ((":" + env["PYTHONPATH"]) if env.get("PYTHONPATH") else ""),
    })
    chk = subprocess.run([sys.executable, "-c", _CHECK_LOADED], cwd=ROOT, env=env, capture_output=True,
                         text=True, timeout=300)
    assert chk.returncode == 0, chk.stdout[-3000:] + chk.stderr[-3000:]
    res = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                          "tests/test_plan.py", "tests/test_oracle.py"],
                         cwd=ROOT, env=env, capture_output=True, text=True, timeout=900)
    log = res.stdout + res.stderr
    assert res.returncode == 0, log[-6000:]
    for marker in ("runtime error:", "AddressSanitizer", "LeakSanitizer"):
        assert marker not in log, log[-6000:]
    assert " passed" in log
