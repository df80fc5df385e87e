"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer (CPU only).

* The oracle (plain C) built with gcc and both sanitizers, LeakSanitizer on,
  and run through every entry point by `sanitize/oracle_main.c`.
* The library's host side -- the C ABI's argument checks, workspace queries
  and workspace carving in `ql_api.cpp` and the allocation-free entry point's
  checks in `ql_scratch.hip` -- compiled with both sanitizers on the host pass
  only (the gfx950 device code is built as always), linked with the other
  objects of the library, and driven by `sanitize/abi_main.cpp` through
  invalid arguments and the evaluated models' descriptors.  No call gets past
  its checks, so no GPU is needed.  LeakSanitizer is off for this run: the HIP
  runtime keeps allocations until the process ends.
First, each sanitizer is shown to report a mistake planted in a small program
of its own, so a silent no-op build cannot pass.
"""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HERE = os.path.join(ROOT, "tests", "sanitize")
ORACLE = os.path.join(ROOT, "oracle")
CSRC = os.path.join(ROOT, "paper_1607_04683_amd", "csrc")
INCLUDE = os.path.join(ROOT, "include")
ROCM = "/opt/rocm"
CLANGXX = os.path.join(ROCM, "llvm", "bin", "clang++")
HIPCC = os.environ.get("HIPCC", os.path.join(ROCM, "bin", "hipcc"))

GCC_SAN = ["-g", "-O1", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
           "-fno-sanitize-recover=all"]
# the host pass of hipcc only: every sanitizer flag behind -Xarch_host
HOST_SAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
            "-Xarch_host", "-fno-sanitize-recover=all", "-Xarch_host", "-fno-omit-frame-pointer"]
LINK_SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all"]


def _run(cmd, env_extra=None, timeout=600):
    env = dict(os.environ, **(env_extra or {}))
    p = subprocess.run(cmd, capture_output=True, text=True, env=env, timeout=timeout)
    return p.returncode, p.stdout + p.stderr


def _need(tool):
    if not (os.path.exists(tool) or shutil.which(tool)):
        pytest.skip(f"{tool} not available")


@pytest.mark.parametrize("kind", ["address", "undefined"])
def test_planted_mistake_is_reported(tmp_path, kind):
    """Each sanitizer alone reports its planted mistake: a heap read one past
    the end (address), a signed overflow (undefined)."""
    _need("gcc")
    src = tmp_path / "bad.c"
    body = {"address": "volatile int *p = malloc(4 * sizeof(int)); int r = p[argc + 3];"
                       " free((void *)p); return r;",
            "undefined": "volatile int x = 2147483647; return x + argc;"}[kind]
    src.write_text("#include <stdlib.h>\nint main(int argc, char **argv) { (void)argv; "
                   + body + " }\n")
    rc, out = _run(["gcc", "-g", "-O1", f"-fsanitize={kind}", "-fno-sanitize-recover=all",
                    str(src), "-o", str(tmp_path / "bad")])
    assert rc == 0, out
    rc, out = _run([str(tmp_path / "bad")])
    want = {"address": "AddressSanitizer: heap-buffer-overflow",
            "undefined": "signed integer overflow"}[kind]
    assert rc != 0 and want in out, out


def test_oracle_under_address_and_undefined_sanitizers(tmp_path):
    _need("gcc")
    exe = tmp_path / "oracle_main"
    rc, out = _run(["gcc", *GCC_SAN, "-std=c11", "-ffp-contract=off", "-fno-fast-math",
                    "-fopenmp", "-I", ORACLE, os.path.join(ORACLE, "qlstm_oracle.c"),
                    os.path.join(HERE, "oracle_main.c"), "-o", str(exe), "-lm"])
    assert rc == 0, out
    rc, out = _run([str(exe)], {"ASAN_OPTIONS": "detect_leaks=1", "OMP_NUM_THREADS": "4"})
    assert rc == 0 and "oracle sanitizer run: ok" in out, out


def _library_objects():
    """The library's objects of a normal build (built here when absent or
    older than a source)."""
    from paper_1607_04683_amd import build
    objdir = os.path.join(os.path.dirname(build.LIB), "_build")
    names = [os.path.splitext(s)[0] + ".o" for s in build.SOURCES]
    if build._stale() or not all(os.path.exists(os.path.join(objdir, n)) for n in names):
        build.build(force=True)
    return build, {n: os.path.join(objdir, n) for n in names}


def test_abi_host_code_under_address_and_undefined_sanitizers(tmp_path):
    _need(HIPCC)
    _need(CLANGXX)
    build, objs = _library_objects()
    san_objs = {}
    for src in ("ql_api.cpp", "ql_scratch.hip"):
        obj = str(tmp_path / (os.path.splitext(src)[0] + ".o"))
        rc, out = _run([HIPCC, "-x", "hip", *build.FLAGS, "-g", *HOST_SAN, "-I", INCLUDE, "-c",
                        os.path.join(CSRC, src), "-o", obj])
        assert rc == 0, out
        san_objs[os.path.splitext(src)[0] + ".o"] = obj
    main_obj = str(tmp_path / "abi_main.o")
    rc, out = _run([CLANGXX, "-std=c++17", "-g", "-O1", *LINK_SAN, "-I", INCLUDE, "-c",
                    os.path.join(HERE, "abi_main.cpp"), "-o", main_obj])
    assert rc == 0, out
    link = [san_objs.get(n, p) for n, p in objs.items()]
    exe = str(tmp_path / "abi_main")
    rc, out = _run([CLANGXX, *LINK_SAN, main_obj, *link, "-L", os.path.join(ROCM, "lib"),
                    "-lamdhip64", "-Wl,-rpath," + os.path.join(ROCM, "lib"), "-o", exe])
    assert rc == 0, out
    rc, out = _run([exe], {"ASAN_OPTIONS": "detect_leaks=0"}, timeout=300)
    assert rc == 0 and "ABI sanitizer run: ok" in out, out
