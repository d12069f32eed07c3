"""CPU: the oracle and the library's host code under AddressSanitizer and
UndefinedBehaviorSanitizer, and a static check of the inline-asm stores.

* The oracle (oracle.c) is rebuilt with gcc's address and undefined-behaviour
  sanitizers and both pin suites run against that build (TC_ORACLE_LIB) in a
  child process with the sanitizer runtime preloaded.
* The library is rebuilt with the host pass sanitized (every -fsanitize
  option applies to the host code alone; the device code is compiled as
  usual) and the host tests (argument checks, the tensor-parallel, reshard and
  cast-item builders against the oracle, the prepared-cast and IPC argument
  checks) run against it (TC_LIB_PATH).  No kernel is launched.
* Each runner first shows that it would catch a bug: a one-byte heap overrun
  in a throwaway library built the same way must abort the child with a
  sanitizer report.
* Every inline-asm store of more than 8 bytes in the device sources ends
  with s_nop 1: the store reads its data registers after issue, a VALU write
  to them needs 2 wait states, and the compiler cannot see into asm.
"""
import glob
import os
import re
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2608_06007_amd", "csrc")
GCC_SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer"]
OVERRUN_C = r"""
#include <stdlib.h>
int overrun(int n) { char* p = (char*)malloc((size_t)n); p[n] = 1; int r = p[0]; free(p); return r; }
"""


def _gcc_runtime():
    libs = []
    for name in ("libasan.so", "libubsan.so"):
        path = subprocess.run(["gcc", f"-print-file-name={name}"], capture_output=True,
                              text=True).stdout.strip()
        if not os.path.isabs(path) or not os.path.exists(path):
            pytest.skip(f"gcc's {name} is not installed")
        libs.append(path)
    return ":".join(libs)


def _clang_runtime():
    found = sorted(glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
    if not found:
        pytest.skip("clang's AddressSanitizer runtime is not installed")
    return found[-1]


def _env(preload, **extra):
    env = dict(os.environ)
    env["LD_PRELOAD"] = preload
    env["ASAN_OPTIONS"] = "detect_leaks=0:abort_on_error=0:halt_on_error=1"
    env["UBSAN_OPTIONS"] = "print_stacktrace=1:halt_on_error=1"
    env.update(extra)
    return env


def _overrun_is_caught(lib_path, preload):
    code = (f"import ctypes; L = ctypes.CDLL({lib_path!r}); "
            "L.overrun.argtypes = [ctypes.c_int]; print(L.overrun(16))")
    r = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True,
                       env=_env(preload), timeout=120)
    return r.returncode != 0 and "AddressSanitizer" in r.stderr


def _run_pytest(files, env, timeout):
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider", *files],
                       cwd=ROOT, capture_output=True, text=True, env=env, timeout=timeout)
    out = r.stdout + r.stderr
    assert "AddressSanitizer" not in out and "runtime error" not in out, out[-4000:]
    assert r.returncode == 0, out[-4000:]
    return out


def test_oracle_pins_under_asan_and_ubsan(tmp_path):
    from oracle import build as obuild
    preload = _gcc_runtime()
    canary = tmp_path / "overrun.c"
    canary.write_text(OVERRUN_C)
    canary_so = str(tmp_path / "liboverrun.so")
    subprocess.run(["gcc", "-O1", "-shared", "-fPIC", *GCC_SAN, "-o", canary_so, str(canary)], check=True)
    assert _overrun_is_caught(canary_so, preload), "the gcc sanitizer runner does not catch an overrun"
    lib = str(tmp_path / "liboracle_san.so")
    cmd = ["gcc", "-O1", "-fno-fast-math", "-std=c11", "-fopenmp", "-shared", "-fPIC", "-Wall",
           *GCC_SAN, "-I", os.path.join(ROOT, "oracle"), "-o", lib,
           os.path.join(ROOT, "oracle", "oracle.c"), "-lm"]
    assert obuild.HERE == os.path.join(ROOT, "oracle")
    subprocess.run(cmd, check=True)
    out = _run_pytest(["tests/test_oracle_fp8.py", "tests/test_oracle_moves.py"],
                      _env(preload, TC_ORACLE_LIB=lib), timeout=900)
    assert " passed" in out


def test_library_host_code_under_asan_and_ubsan(tmp_path):
    from paper_2608_06007_amd import build as lbuild
    preload = _clang_runtime()
    canary = tmp_path / "overrun.c"
    canary.write_text(OVERRUN_C)
    canary_so = str(tmp_path / "liboverrun.so")
    subprocess.run([lbuild.HIPCC, "-x", "c", "-O1", "-shared", "-fPIC", "-fsanitize=address,undefined",
                    "-fno-sanitize-recover=undefined", "-o", canary_so, str(canary)], check=True)
    assert _overrun_is_caught(canary_so, preload), "the clang sanitizer runner does not catch an overrun"
    lib = lbuild.build(sanitize=True, out=str(tmp_path / "libtchip_san.so"))
    out = _run_pytest(["tests/test_library_host.py"], _env(preload, TC_LIB_PATH=lib), timeout=900)
    assert " passed" in out


# ---------------------------------------------------------------------------

# store instructions that read more than 8 bytes of data registers
WIDE_STORES = re.compile(r"\b(global|flat|buffer|scratch)_store_(dwordx3|dwordx4|b96|b128)\b")


def _asm_statements(text):
    """The instruction template of every asm(...) statement: its string
    literals before the first operand colon, joined."""
    out = []
    for m in re.finditer(r"\basm\s+(volatile\s*)?\(", text):
        i, parts = m.end(), []
        while True:
            lit = re.compile(r'\s*"((?:[^"\\]|\\.)*)"').match(text, i)
            if not lit:
                break
            parts.append(lit.group(1))
            i = lit.end()
        out.append("".join(parts))
    return out


def test_wide_inline_asm_stores_end_with_two_wait_states():
    found = 0
    for path in sorted(glob.glob(os.path.join(CSRC, "*.hip")) + glob.glob(os.path.join(CSRC, "*.h"))):
        for stmt in _asm_statements(open(path).read()):
            if not WIDE_STORES.search(stmt):
                continue
            found += 1
            instrs = [s.strip() for s in stmt.replace("\\n", "\n").replace("\\t", " ").split("\n") if s.strip()]
            last_store = max(k for k, s in enumerate(instrs) if WIDE_STORES.search(s))
            tail = instrs[last_store + 1:]
            assert tail and re.fullmatch(r"s_nop\s+([1-9]|1[0-5])", tail[0]), \
                f"{os.path.basename(path)}: wide asm store without s_nop after it: {stmt!r}"
    assert found >= 2, "the check found no wide asm stores: the pattern no longer matches the sources"


def test_the_asm_check_rejects_a_store_without_wait_states():
    bad = 'asm volatile("global_store_dwordx4 %0, %1, off sc1" ::"v"(p), "v"(v) : "memory");'
    good = 'asm volatile("global_store_dwordx4 %0, %1, off sc1\\n\\ts_nop 1" ::"v"(p), "v"(v) : "memory");'
    for stmt, ok in ((_asm_statements(bad)[0], False), (_asm_statements(good)[0], True)):
        instrs = [s.strip() for s in stmt.replace("\\n", "\n").replace("\\t", " ").split("\n") if s.strip()]
        tail = instrs[max(k for k, s in enumerate(instrs) if WIDE_STORES.search(s)) + 1:]
        assert bool(tail and re.fullmatch(r"s_nop\s+([1-9]|1[0-5])", tail[0])) == ok
