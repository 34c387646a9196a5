"""Build the gfx950 HIP library libapex_decode.so in-tree with hipcc."""
import os
import subprocess
import sys
import tempfile

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libapex_decode.so")
SOURCES = [os.path.join(CSRC, "apex_decode.hip"), os.path.join(CSRC, "kv_append.hip"),
           os.path.join(CSRC, "plan_host.cpp"), os.path.join(CSRC, "status.cpp")]
CPU_LIB = os.path.join(HERE, "libapex_cpu.so")
CPU_DIR = os.path.join(CSRC, "cpu")
OVERLAP_LIB = os.path.join(HERE, "libapex_overlap.so")
OVERLAP_SOURCES = [os.path.join(CSRC, "overlap", "overlap.hip")]
TRACE_LIB = os.path.join(HERE, "libapex_decode_trace.so")
PROBE_LIB = os.path.join(HERE, "libapex_hbm_probe.so")
PROBE_SOURCES = [os.path.join(CSRC, "hbm_probe.hip")]
HEADERS = [os.path.join(ROOT, "include", "apex_decode.h"),
           os.path.join(ROOT, "include", "apex_kv_append.h"),
           os.path.join(ROOT, "include", "apex_decode_trace.h"),
           os.path.join(CSRC, "kernels.h"), os.path.join(CSRC, "plan_policy.h"),
           os.path.join(CSRC, "status.h")]

HIPCC_FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
    "-Wall", "-Wno-unused-function",
    # packed fp32 VALU forms stay off (compiler emits plain fp32 ops instead)
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I", os.path.join(ROOT, "include"), "-I", CSRC,
]


def _compile(sources, out, extra, quiet):
    hipcc = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
    cmd = [hipcc, *HIPCC_FLAGS, *extra, *sources, "-o", out + ".tmp"]
    if not quiet:
        print(" ".join(cmd), flush=True)
    subprocess.check_call(cmd)
    os.replace(out + ".tmp", out)
    return out


CXX_FLAGS = ["-O3", "-std=c++17", "-fPIC", "-fvisibility=hidden", "-Wall", "-Wextra", "-Wno-unused-parameter",
             "-I", os.path.join(ROOT, "include"), "-I", CPU_DIR]
ISA_FLAGS = {
    "simd_avx512": ["-mavx512f", "-mavx512bw", "-mavx512vl", "-mavx512dq", "-mf16c", "-mfma"],
    "simd_avx2": ["-mavx2", "-mfma", "-mf16c"],
}


def _run(cmd, quiet):
    if not quiet:
        print(" ".join(cmd), flush=True)
    subprocess.check_call(cmd)


def build_cpu(out=CPU_LIB, quiet=False):
    """Compile the host paged-attention backend (g++, baseline x86-64 host
    code plus one object per SIMD instruction set)."""
    cxx = os.environ.get("CXX", "g++")
    with tempfile.TemporaryDirectory() as tmp:
        objs = []
        for ns, flags in ISA_FLAGS.items():
            obj = os.path.join(tmp, f"attend_{ns}.o")
            _run([cxx, *CXX_FLAGS, *flags, f"-DAPEX_SIMD_NS={ns}", "-c",
                  os.path.join(CPU_DIR, "attend_simd.cpp"), "-o", obj], quiet)
            objs.append(obj)
        _run([cxx, *CXX_FLAGS, "-shared", "-pthread", os.path.join(CPU_DIR, "cpu_attention.cpp"),
              os.path.join(CSRC, "sched", "scheduler.cpp"), *objs, "-o", out + ".tmp"], quiet)
    os.replace(out + ".tmp", out)
    return out


def build(out=LIB, extra=(), quiet=False):
    """Compile the decode-attention library, its work-group trace build (the
    same sources with APEX_TRACE_WORK_GROUPS), the host attention backend,
    the overlap runtime (linked against the host backend) and the HBM probe
    library."""
    build_cpu(quiet=quiet)
    _compile(PROBE_SOURCES, PROBE_LIB, extra, quiet)
    _compile(SOURCES, TRACE_LIB, [*extra, "-DAPEX_TRACE_WORK_GROUPS"], quiet)
    _compile(OVERLAP_SOURCES, OVERLAP_LIB,
             [*extra, "-L", HERE, "-lapex_cpu", "-Wl,-rpath,$ORIGIN", "-pthread"], quiet)
    return _compile(SOURCES, out, extra, quiet)


if __name__ == "__main__":
    build()
    sys.exit(0)
