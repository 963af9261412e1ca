"""Host-side sanitizer runs (CPU only).

The oracle is built with gcc under AddressSanitizer and UndefinedBehaviour-
Sanitizer (leak checking on) and driven through every entry point on small
requests with exact-size buffers (tests/native/oracle_asan_driver.c).  The
codec library's host code (skv_api.cpp: validation, plans, geometry, grouped
and upgrade sizes, argument checks of the device calls) is rebuilt with the
same sanitizers on the host side only and linked with the regular device
objects; its driver (tests/native/lib_asan_driver.cpp) touches no device.
"""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
NATIVE = os.path.join(ROOT, "tests", "native")


def _run(exe, env_extra):
    env = dict(os.environ, **env_extra)
    res = subprocess.run([exe], capture_output=True, text=True, timeout=600, env=env)
    assert res.returncode == 0, res.stdout[-2000:] + res.stderr[-4000:]
    assert res.stdout.startswith("ok"), res.stdout
    return res


def test_oracle_clean_under_asan_ubsan(tmp_path):
    gcc = shutil.which("gcc")
    if gcc is None:
        pytest.skip("gcc not found")
    exe = str(tmp_path / "oracle_asan")
    flags = ["-O1", "-g", "-std=c11", "-ffp-contract=off", "-fno-fast-math", "-fno-omit-frame-pointer",
             "-fsanitize=address,undefined", "-fno-sanitize-recover=all"]
    srcs = [os.path.join(ROOT, "oracle", "skv_oracle.c"), os.path.join(NATIVE, "oracle_asan_driver.c")]
    subprocess.run([gcc, *flags, *srcs, "-o", exe, "-lm"], check=True, capture_output=True, timeout=300)
    _run(exe, {"ASAN_OPTIONS": "detect_leaks=1"})


def test_library_host_code_clean_under_asan_ubsan(tmp_path):
    from paper_2606_08635_amd import build as B

    if not os.path.exists(B.HIPCC):
        pytest.skip("hipcc not found")
    objs = [os.path.join(B.BUILD_DIR, os.path.splitext(s)[0] + ".o") for s in B.SOURCES if s != "skv_api.cpp"]
    if not all(os.path.exists(o) for o in objs):
        B.build()
    # host-side instrumentation only: every sanitizer flag is scoped to the host pass
    host = []
    for f in ("-fsanitize=address", "-fsanitize=undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer", "-g"):
        host += ["-Xarch_host", f]
    api, drv, exe = (str(tmp_path / x) for x in ("skv_api.o", "driver.o", "lib_asan"))
    for src, obj in ((os.path.join(B.CSRC, "skv_api.cpp"), api), (os.path.join(NATIVE, "lib_asan_driver.cpp"), drv)):
        r = subprocess.run([B.HIPCC, *B.FLAGS, *host, "-c", src, "-o", obj], capture_output=True, text=True, timeout=600)
        assert r.returncode == 0, r.stderr[-3000:]
    r = subprocess.run([B.HIPCC, "--offload-arch=gfx950", *host, "-o", exe, drv, api, *objs],
                       capture_output=True, text=True, timeout=600)
    assert r.returncode == 0, r.stderr[-3000:]
    # the HIP runtime keeps allocations alive at exit: leak checking off for this binary
    _run(exe, {"ASAN_OPTIONS": "detect_leaks=0"})
