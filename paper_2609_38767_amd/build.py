"""Build libdattri.so for gfx950 with hipcc (in-tree; no JIT cache).

    python -m paper_2609_38767_amd.build             # the library
    python -m paper_2609_38767_amd.build --sanitize  # host checks (CPU only)

Every source under csrc/ is compiled to an object under _build/ in parallel and
linked into paper_2609_38767_amd/libdattri.so.

--sanitize builds a second library, _build/asan/libdattri.so, whose host code
(the C ABI, planner, generator and calibration reader: the .cpp sources) is
instrumented with AddressSanitizer and UndefinedBehaviorSanitizer; device code
is built as usual and carries no instrumentation.  It is for the host-only
tests: load it with DATTRI_LIB pointing at it and the sanitizer runtime
preloaded, e.g.

    LD_PRELOAD=$(/opt/rocm/llvm/bin/clang -print-file-name=libclang_rt.asan-x86_64.so) \
    ASAN_OPTIONS=detect_leaks=0 UBSAN_OPTIONS=halt_on_error=1:print_stacktrace=1 \
    DATTRI_LIB=_build/asan/libdattri.so python -m pytest tests -m "not gpu"
"""
import concurrent.futures as cf
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
BUILD = os.path.join(ROOT, "_build")
LIB = os.path.join(HERE, "libdattri.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"

COMMON = ["-O3", "-std=c++17", "-fPIC", "-Wall", "-Werror", "-Wno-unused-function",
          "-I", os.path.join(ROOT, "include"), "-I", CSRC]
# Device code: gfx950 only; packed-FP32 instruction selection disabled.
DEVICE = [f"--offload-arch={ARCH}", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
          "-Wno-unused-command-line-argument"]


def sources():
    return sorted(f for f in os.listdir(CSRC) if f.endswith((".hip", ".cpp")))


# Host-code sanitizers (each flag after -Xarch_host: host code only).
SANITIZE = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
            "-Xarch_host", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer", "-g"]


def _compile(src, build_dir=BUILD, sanitize=False):
    obj = os.path.join(build_dir, src + ".o")
    cmd = [HIPCC] + COMMON
    if src.endswith(".hip"):
        cmd += DEVICE + ["-x", "hip"]
    elif sanitize:
        cmd += SANITIZE
    cmd += ["-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    # hipcc's host pass warns that it does not know the packed-fp32 feature
    err = "\n".join(l for l in r.stderr.splitlines() if "packed-fp32-ops" not in l)
    if r.returncode != 0:
        raise RuntimeError(f"compile failed: {src}\n{' '.join(cmd)}\n{err}")
    return obj


def build(jobs=None, sanitize=False):
    build_dir = os.path.join(BUILD, "asan") if sanitize else BUILD
    lib = os.path.join(build_dir, "libdattri.so") if sanitize else LIB
    os.makedirs(build_dir, exist_ok=True)
    srcs = sources()
    jobs = jobs or min(len(srcs), os.cpu_count() or 4, 16)
    with cf.ThreadPoolExecutor(jobs) as ex:
        objs = list(ex.map(lambda src: _compile(src, build_dir, sanitize), srcs))
    tmp = lib + ".tmp"
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp] + objs
    if sanitize:  # the runtime comes from the preloaded sanitizer library
        cmd += ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined", "-shared-libsan"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed\n{' '.join(cmd)}\n{r.stderr}")
    os.replace(tmp, lib)
    return lib


if __name__ == "__main__":
    print(build(sanitize="--sanitize" in sys.argv[1:]))
    sys.exit(0)
