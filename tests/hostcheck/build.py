"""Builds the host-side bounds checker (test infrastructure): the library's
own sources (csrc/*.hip, api.cpp) plus tests/hostcheck/*.cpp, with
AddressSanitizer and UndefinedBehaviorSanitizer on the host code only, into
tests/hostcheck/_build/hostcheck.  The kernels' device code is compiled too
(the host code registers it) but never runs: the checker installs a launch
observer that receives every launch instead of a GPU.  The build is reused
while no source changed (hash of the sources and flags)."""
from __future__ import annotations

import concurrent.futures
import hashlib
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
CSRC = os.path.join(ROOT, "paper_2507_01040_amd", "csrc")
OUT = os.path.join(HERE, "_build")
EXE = os.path.join(OUT, "hostcheck")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
LIB_SOURCES = ["api.cpp", "conv_mfma.hip", "conv1d_mfma.hip", "conv_direct.hip", "act.hip",
               "block_small.hip", "block_noalloc.hip", "linear_mfma.hip", "mfma_probe.hip"]
CHECK_SOURCES = ["check_main.cpp", "check_conv_mfma.cpp", "check_conv1d.cpp", "check_block_small.cpp",
                 "check_act.cpp", "check_linear.cpp", "check_direct.cpp",
                 "check_generic.cpp"]
# sanitizers on the host side only; each -fsanitize= behind -Xarch_host
FLAGS = ["--offload-arch=gfx950", "-O2", "-g", "-std=c++17", "-fPIC", "-fno-omit-frame-pointer",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-I" + os.path.join(ROOT, "include"), "-I" + CSRC, "-I" + HERE,
         "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
         "-Xarch_host", "-fno-sanitize-recover=undefined"]
LINK = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
        "-L/opt/rocm/lib", "-lamdhip64"]


def _sources():
    srcs = [os.path.join(CSRC, s) for s in LIB_SOURCES]
    srcs += [os.path.join(HERE, s) for s in CHECK_SOURCES]
    hdrs = [os.path.join(CSRC, h) for h in sorted(os.listdir(CSRC)) if h.endswith(".hpp")]
    hdrs += [os.path.join(HERE, "check.hpp"), os.path.join(ROOT, "include", "cliffconv.h")]
    return srcs, hdrs


def _digest(paths):
    h = hashlib.sha256(" ".join(FLAGS + LINK).encode())
    for p in paths:
        with open(p, "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def build(force: bool = False) -> str:
    srcs, hdrs = _sources()
    digest = _digest(srcs + hdrs)
    stamp = os.path.join(OUT, "digest")
    if not force and os.path.exists(EXE) and os.path.exists(stamp):
        with open(stamp) as f:
            if f.read().strip() == digest:
                return EXE
    os.makedirs(OUT, exist_ok=True)

    def compile_one(src):
        obj = os.path.join(OUT, os.path.basename(src) + ".o")
        r = subprocess.run([HIPCC, *FLAGS, "-c", src, "-o", obj], capture_output=True, text=True)
        if r.returncode:
            raise RuntimeError("hostcheck compile failed: %s\n%s" % (src, r.stderr[-4000:]))
        return obj

    with concurrent.futures.ThreadPoolExecutor(max_workers=min(8, len(srcs))) as ex:
        objs = list(ex.map(compile_one, srcs))
    tmp = EXE + ".tmp%d" % os.getpid()
    r = subprocess.run([HIPCC, *objs, "-o", tmp, *LINK], capture_output=True, text=True)
    if r.returncode:
        raise RuntimeError("hostcheck link failed\n%s" % r.stderr[-4000:])
    os.replace(tmp, EXE)
    with open(stamp, "w") as f:
        f.write(digest)
    return EXE


def run(lines, timeout=600):
    """Runs the checker over case lines; returns its output lines."""
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:abort_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    r = subprocess.run([build()], input="\n".join(lines) + "\n", capture_output=True, text=True,
                       env=env, timeout=timeout)
    if r.returncode:
        raise RuntimeError("hostcheck exited with %d\n%s" % (r.returncode, r.stderr[-6000:]))
    return r.stdout.strip().split("\n")


if __name__ == "__main__":
    print(build(force=True))
