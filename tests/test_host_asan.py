"""AddressSanitizer over the host side of the C ABI (no GPU).

tests/asan_api_driver.cpp calls every entry point's validation path and the
workspace sizing over the whole shape set (all d, d_v, m, variants, lengths,
segment counts and chunk lengths), each call with at least one invalid argument
so that no kernel is launched.  The ABI's host code (flex_api.hip: validation,
shape set, frequency groups, value-width padding, segment heuristics, the
scratch table) is compiled with -fsanitize=address for the host only; the
kernels' objects are the library's own build.  Any out-of-bounds access, use
after free or other ASan finding in those paths fails the test.
"""
import os
import subprocess
import tempfile

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
CLANGXX = "/opt/rocm/llvm/bin/clang++"
KERNEL_SOURCES = ["flex_fwd", "flex_bwd", "flex_bwd_dq", "flex_decode", "flex_awd"]


def _kernel_objects():
    from paper_2606_27748_amd import build as B
    objs = [os.path.join(B.BUILD, s + ".o") for s in KERNEL_SOURCES]
    if not all(os.path.exists(o) for o in objs):
        B.build()
    return objs


@pytest.mark.skipif(not (os.path.exists(HIPCC) and os.path.exists(CLANGXX)), reason="needs hipcc and clang++")
def test_host_abi_under_asan():
    objs = _kernel_objects()
    inc = os.path.join(ROOT, "include")
    with tempfile.TemporaryDirectory() as tmp:
        api = os.path.join(tmp, "flex_api_asan.o")
        drv = os.path.join(tmp, "driver.o")
        exe = os.path.join(tmp, "asan_api_driver")
        # host side only: each -fsanitize= is given to the host compilation
        subprocess.run([HIPCC, "--offload-arch=gfx950", "-O1", "-g", "-std=c++17", "-fPIC",
                        "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
                        "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fno-omit-frame-pointer",
                        "-I", inc, "-c", os.path.join(ROOT, "paper_2606_27748_amd", "csrc", "flex_api.hip"),
                        "-o", api], check=True, capture_output=True)
        subprocess.run([CLANGXX, "-std=c++17", "-O1", "-g", "-fsanitize=address", "-fno-omit-frame-pointer",
                        "-I", inc, "-c", os.path.join(ROOT, "tests", "asan_api_driver.cpp"), "-o", drv],
                       check=True, capture_output=True)
        subprocess.run([CLANGXX, "-fsanitize=address", drv, api] + objs +
                       ["-L/opt/rocm/lib", "-lamdhip64", "-Wl,-rpath,/opt/rocm/lib", "-o", exe],
                       check=True, capture_output=True)
        env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:abort_on_error=0:halt_on_error=1")
        r = subprocess.run([exe], capture_output=True, text=True, timeout=300, env=env)
        assert r.returncode == 0 and r.stdout.strip().endswith("ok"), (r.returncode, r.stdout[-2000:],
                                                                       r.stderr[-4000:])
