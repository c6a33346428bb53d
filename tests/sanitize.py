"""Host sanitizer runs (no GPU needed).

1. The oracle (``oracle/oracle.c``) built by gcc with AddressSanitizer and
   UndefinedBehaviorSanitizer; every pin of ``tests/pins.py`` runs against
   that build in a child process with gcc's runtime preloaded.
2. The HIP library built with AddressSanitizer on its host code only (each
   sanitizer flag behind ``-Xarch_host``; the device code is built as usual),
   into a separate directory; the C-ABI checks of ``tests/test_abi.py`` run
   against that build in a child process with clang's runtime preloaded.

Run ``python tests/sanitize.py``: exit status 0 when both runs are clean.
The builds go to ``_build_sanitize/`` beside this file's repository root
(outside the package) and are redone only when a source is newer.
"""
from __future__ import annotations

import glob
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
OUT = os.path.join(ROOT, "_build_sanitize")
CSRC = os.path.join(ROOT, "paper_1805_02867_amd", "csrc")
INCLUDE = os.path.join(ROOT, "include")
ORACLE_SRC = os.path.join(ROOT, "oracle", "oracle.c")
ORACLE_LIB = os.path.join(OUT, "liboracle_asan.so")
OSM_LIB = os.path.join(OUT, "libosoftmax_hostasan.so")
ASAN_OPTIONS = "detect_leaks=0:abort_on_error=0:halt_on_error=1:exitcode=23"
UBSAN_OPTIONS = "print_stacktrace=1:halt_on_error=1:exitcode=24"


def _stale(out: str, srcs: list[str]) -> bool:
    if not os.path.exists(out):
        return True
    t = os.path.getmtime(out)
    return any(os.path.getmtime(s) > t for s in srcs)


def build_oracle() -> str:
    if _stale(ORACLE_LIB, [ORACLE_SRC]):
        os.makedirs(OUT, exist_ok=True)
        subprocess.check_call([
            "gcc", "-O1", "-g", "-fno-omit-frame-pointer", "-ffp-contract=off",
            "-fno-fast-math", "-fopenmp", "-fsanitize=address,undefined",
            "-fno-sanitize-recover=undefined", "-shared", "-fPIC", ORACLE_SRC,
            "-o", ORACLE_LIB, "-lm"])
    return ORACLE_LIB


def _hipcc() -> str:
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    return os.path.join(rocm, "bin", "hipcc")


def build_library() -> str:
    srcs = sorted(glob.glob(os.path.join(CSRC, "*.hip")))
    deps = srcs + glob.glob(os.path.join(CSRC, "*.h*")) + glob.glob(os.path.join(INCLUDE, "*.h"))
    if not _stale(OSM_LIB, deps):
        return OSM_LIB
    objdir = os.path.join(OUT, "obj")
    os.makedirs(objdir, exist_ok=True)
    host_asan = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fno-omit-frame-pointer"]
    flags = ["--offload-arch=gfx950", "-O1", "-g", "-std=c++17", "-fPIC",
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
             "-fvisibility=hidden", "-Wno-unused-command-line-argument",
             f"-I{INCLUDE}", f"-I{CSRC}", *host_asan]
    procs, objs = [], []
    for s in srcs:
        o = os.path.join(objdir, os.path.basename(s)[:-4] + ".o")
        objs.append(o)
        procs.append(subprocess.Popen([_hipcc(), *flags, "-c", s, "-o", o],
                                      stdout=subprocess.PIPE, stderr=subprocess.STDOUT))
    for p in procs:
        out, _ = p.communicate()
        if p.returncode != 0:
            sys.stderr.write(out.decode(errors="replace"))
            raise RuntimeError("host-sanitized build failed")
    subprocess.check_call([_hipcc(), "--offload-arch=gfx950", "-shared", "-fPIC",
                           "-Xarch_host", "-fsanitize=address", *objs, "-o", OSM_LIB])
    return OSM_LIB


def _clang_asan_runtime() -> str:
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    hits = glob.glob(os.path.join(rocm, "llvm", "lib", "clang", "*", "lib", "linux",
                                  "libclang_rt.asan-x86_64.so"))
    if not hits:
        raise RuntimeError("clang's ASan runtime not found")
    return hits[0]


def _gcc_runtime(name: str) -> str:
    return subprocess.check_output(["gcc", f"-print-file-name={name}"], text=True).strip()


def _child(code: str, preload: str) -> subprocess.CompletedProcess:
    env = dict(os.environ)
    env["LD_PRELOAD"] = preload
    env["ASAN_OPTIONS"] = ASAN_OPTIONS
    env["UBSAN_OPTIONS"] = UBSAN_OPTIONS
    env["PYTHONPATH"] = os.pathsep.join([ROOT, HERE, env.get("PYTHONPATH", "")])
    return subprocess.run([sys.executable, "-c", code], cwd=ROOT, env=env,
                          capture_output=True, text=True)


ORACLE_CHILD = """
import oracle, pins
orc = oracle.load({lib!r})
for check in pins.ALL:
    check(orc)
print("oracle pins passed:", len(pins.ALL))
"""

ABI_CHILD = """
import sys, pytest
import paper_1805_02867_amd as osm
osm.LIB_PATH = {lib!r}
osm._lib = None
rc = pytest.main(["-q", "-p", "no:cacheprovider", "-m", "not gpu", {test!r}])
assert osm.lib()._name == {lib!r}
sys.exit(int(rc))
"""


def sanitizer_report(text: str) -> bool:
    return "AddressSanitizer" in text or "runtime error:" in text or "LeakSanitizer" in text


def instrumented(lib: str) -> bool:
    """The build calls into the ASan runtime (its checks are really there)."""
    syms = subprocess.check_output(["nm", "-D", "--undefined-only", lib], text=True)
    return "__asan_report_load" in syms or "__asan_load" in syms


def run() -> int:
    status = 0
    lib = build_oracle()
    if not instrumented(lib):
        print("oracle build carries no ASan checks")
        return 1
    pre = " ".join([_gcc_runtime("libasan.so"), _gcc_runtime("libubsan.so")])
    r = _child(ORACLE_CHILD.format(lib=lib), pre)
    print("== oracle (gcc, address + undefined):", "rc", r.returncode)
    print((r.stdout + r.stderr)[-3000:])
    if r.returncode != 0 or sanitizer_report(r.stdout + r.stderr):
        status = 1
    lib = build_library()
    if not instrumented(lib):
        print("library build carries no host ASan checks")
        return 1
    r = _child(ABI_CHILD.format(lib=lib, test=os.path.join(HERE, "test_abi.py")),
               _clang_asan_runtime())
    print("== library host code (clang, address):", "rc", r.returncode)
    print((r.stdout + r.stderr)[-3000:])
    if r.returncode != 0 or sanitizer_report(r.stdout + r.stderr):
        status = 1
    return status


if __name__ == "__main__":
    sys.exit(run())
