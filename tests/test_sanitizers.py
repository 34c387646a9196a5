"""The library's host code under sanitizers (CPU only, no GPU).

tests/sanitize/driver.cpp runs seeded random cases through the fp64 oracle,
the host paged-attention backend (compared with the oracle), the partition's
host mirror (against an explicit line of positions) and the strategy
selection.  It is built with g++ twice: with AddressSanitizer +
UndefinedBehaviorSanitizer over all of them, and with ThreadSanitizer over the
host backend and its thread pool (several thread counts, pool resizes,
chunked pairs).  Any sanitizer report or failed check fails the test.
"""
import os
import shutil
import subprocess
import tempfile
from concurrent.futures import ThreadPoolExecutor

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2506_03296_amd", "csrc")
INC = ["-I", os.path.join(ROOT, "include"), "-I", CSRC, "-I", os.path.join(CSRC, "cpu")]
# plan_policy.h includes the HIP runtime header for its __host__ __device__
# markers; with g++ they expand to nothing
HIP_HOST = ["-I", "/opt/rocm/include", "-D__HIP_PLATFORM_AMD__"]
ISA = {"simd_avx512": ["-mavx512f", "-mavx512bw", "-mavx512vl", "-mavx512dq", "-mf16c", "-mfma"],
       "simd_avx2": ["-mavx2", "-mfma", "-mf16c"]}
SAN = {"asan": ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer"],
       "tsan": ["-fsanitize=thread"]}


def _have(tool):
    return shutil.which(tool) is not None


def _build(kind, tmp):
    san = SAN[kind]
    flags = ["-O1", "-g", *san]
    jobs = []
    # the oracle: instrumented under ASan/UBSan; under TSan it runs single-threaded, uninstrumented
    jobs.append(["gcc", "-std=c11", "-fopenmp", "-O1", "-g", *(san if kind == "asan" else []), "-c",
                 os.path.join(ROOT, "oracle", "ref_decode.c"), "-o", os.path.join(tmp, "oracle.o")])
    for ns, isa in ISA.items():
        jobs.append(["g++", "-std=c++17", *flags, *isa, *INC, f"-DAPEX_SIMD_NS={ns}", "-c",
                     os.path.join(CSRC, "cpu", "attend_simd.cpp"), "-o", os.path.join(tmp, f"{ns}.o")])
    for src in (os.path.join(CSRC, "cpu", "cpu_attention.cpp"), os.path.join(CSRC, "sched", "scheduler.cpp"),
                os.path.join(CSRC, "plan_host.cpp"), os.path.join(CSRC, "status.cpp"),
                os.path.join(ROOT, "tests", "sanitize", "driver.cpp")):
        obj = os.path.join(tmp, os.path.basename(src) + ".o")
        jobs.append(["g++", "-std=c++17", *flags, "-mf16c", *INC, *HIP_HOST, "-c", src, "-o", obj])
    with ThreadPoolExecutor(max_workers=4) as ex:
        for r in ex.map(lambda c: subprocess.run(c, capture_output=True, text=True), jobs):
            assert r.returncode == 0, r.stderr[-3000:]
    objs = [j[j.index("-o") + 1] for j in jobs]
    exe = os.path.join(tmp, f"driver_{kind}")
    r = subprocess.run(["g++", *san, "-fopenmp", "-pthread", *objs, "-o", exe, "-lm"], capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-3000:]
    return exe


def _supported(kind):
    """The compiler and its sanitizer runtime work on this host."""
    if not (_have("gcc") and _have("g++")):
        return False
    with tempfile.TemporaryDirectory() as tmp:
        src = os.path.join(tmp, "t.cpp")
        open(src, "w").write("int main() { return 0; }\n")
        exe = os.path.join(tmp, "t")
        if subprocess.run(["g++", *SAN[kind], src, "-o", exe], capture_output=True).returncode != 0:
            return False
        return subprocess.run([exe], capture_output=True).returncode == 0


def _cpu_has_avx2():
    try:
        flags = open("/proc/cpuinfo").read()
    except OSError:
        return False
    return all(f in flags for f in ("avx2", "fma", "f16c"))


@pytest.mark.parametrize("kind,mode,cases", [("asan", "all", 60), ("tsan", "threads", 40)])
def test_host_code_under_sanitizers(kind, mode, cases):
    if not _cpu_has_avx2():
        pytest.skip("the host backend needs AVX2 + FMA + F16C")
    if not _supported(kind):
        pytest.skip(f"{kind} is not available with this compiler")
    with tempfile.TemporaryDirectory() as tmp:
        exe = _build(kind, tmp)
        env = dict(os.environ)
        # verify_asan_link_order=0: a library the environment preloads may
        # come before the ASan runtime; that is fine for this driver
        env["ASAN_OPTIONS"] = "detect_leaks=1:abort_on_error=0:halt_on_error=1:verify_asan_link_order=0"
        env["UBSAN_OPTIONS"] = "print_stacktrace=1:halt_on_error=1"
        env["TSAN_OPTIONS"] = "halt_on_error=1:second_deadlock_stack=1"
        r = subprocess.run([exe, str(cases), mode], capture_output=True, text=True, env=env, timeout=600)
        report = r.stdout[-2000:] + r.stderr[-6000:]
        print(report)
        assert r.returncode == 0, report
        for marker in ("AddressSanitizer", "runtime error", "ThreadSanitizer", "LeakSanitizer"):
            assert marker not in r.stderr, report
        assert f"{cases} cases, 0 failures" in r.stdout
