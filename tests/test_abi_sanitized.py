"""The C ABI's host code under AddressSanitizer and UBSan, on the CPU: the library's sources
are built with both sanitizers on their host side only (each -fsanitize behind -Xarch_host;
the device code is built as usual and never run), linked with the HIP runtime, and driven
by tests/abi_sanitize_driver.cpp:
every entry point with arguments that must fail validation, the host-only helpers at their
edges, offsets and shapes that would overflow careless size arithmetic, and (when the runtime
sees no device) well-formed calls, whose host-side layouts and offset tables all run before
the first runtime call fails.  Any invalid memory access, signed overflow, out-of-range
conversion or other undefined behaviour aborts the driver.  Skipped where a GPU is visible:
the driver's fake device pointers are for a runtime that has no device."""
import concurrent.futures as cf
import os
import subprocess

import pytest
import torch

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2608_03276_amd", "csrc")
CLANG = "/opt/rocm/llvm/bin/clang++"
ROCM = "/opt/rocm"
SOURCES = ["abi.cpp", "guide_scores.hip", "guide_attention.hip", "quantize.hip", "select.hip", "compact.hip"]
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer"]
HOST_SAN = [x for f in SAN for x in ("-Xarch_host", f)]  # host code only

pytestmark = [pytest.mark.skipif(not os.path.exists(CLANG), reason="the ROCm clang is not installed"),
              pytest.mark.skipif(torch.cuda.device_count() > 0, reason="fake device pointers; run where no GPU is visible")]


def _run(cmd, **kw):
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True, **kw)
    return r.returncode, r.stdout


def test_abi_host_code_under_sanitizers(tmp_path):
    inc = ["-I", os.path.join(ROOT, "include"), "-I", os.path.join(ROCM, "include")]
    jobs = []
    for src in SOURCES:
        obj = str(tmp_path / (os.path.splitext(src)[0] + ".o"))
        jobs.append(([CLANG, "-x", "hip", "--offload-arch=gfx950", "-O1", "-g", "-std=c++17", *HOST_SAN, *inc,
                      "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops", "-c", os.path.join(CSRC, src), "-o", obj],
                     obj))
    drv = str(tmp_path / "driver.o")
    jobs.append(([CLANG, "-x", "c++", "-O1", "-g", "-std=c++17", *SAN, *inc, "-D__HIP_PLATFORM_AMD__", "-c",
                  os.path.join(ROOT, "tests", "abi_sanitize_driver.cpp"), "-o", drv], drv))
    with cf.ThreadPoolExecutor(max_workers=4) as ex:
        for (cmd, _), (rc, out) in zip(jobs, ex.map(lambda j: _run(j[0]), jobs)):
            assert rc == 0, f"{' '.join(cmd)}\n{out}"
    exe = str(tmp_path / "abi_driver")
    rc, out = _run([CLANG, *SAN, *[o for _, o in jobs], "-L", os.path.join(ROCM, "lib"), "-lamdhip64",
                    f"-Wl,-rpath,{os.path.join(ROCM, 'lib')}", "-o", exe])
    assert rc == 0, out
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:halt_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    rc, out = _run([exe], env=env, timeout=300)
    print(out)
    assert rc == 0, out
    assert " 0 failures" in out, out
