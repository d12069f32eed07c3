"""The oracle's pins catch plausible mistakes (CPU only).

Each mutant is oracle.c with one deliberate, plausible error: a wrong tie
rule, wrong saturation, wrong subnormal magnitudes, a dropped zero sign, a
signed amax, a wrong scale constant, the wrong code for a non-finite tile,
a transposed (column-major) scale grid in the cast or in its inverse, a
ties-away bf16
rounding, a short copy, a gather that strides by the block size, or a
digest weight off by one.  Each is compiled with the oracle's own flags and
the pin suites run against it in a subprocess; a mutant that no pin fails
would mean the pins do not pin that part of the oracle.  Every mutant stays
inside its buffers (a transposed grid is stored densely column-major, not
with the row pitch), so a caught mutant fails a test rather than corrupting
the heap of the pytest process that runs the pins.
"""
import concurrent.futures as cf
import os
import subprocess
import sys

import pytest

from oracle import build as oracle_build

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
FP8 = "tests/test_oracle_fp8.py"
MOVES = "tests/test_oracle_moves.py"

# name: (text in oracle.c, replacement, pin suite expected to fail)
MUTANTS = {
    "tie_rule": ("code = (lo & 1) ? hi : lo;", "code = hi;", FP8),
    "saturation": ("return sign | E4M3_MAX_CODE; /* satfinite */", "return sign | 0x7F; /* satfinite */", FP8),
    "subnormal_magnitude": ("if (e == 0) return ldexp((double)m, -9);",
                            "if (e == 0) return ldexp((double)m, -10);", FP8),
    "zero_sign": ("q[r * q_ld + c] = (x[r * ld + c] & 0x8000u) ? 0x80 : 0x00;",
                  "q[r * q_ld + c] = 0x00;", FP8),
    "signed_amax": ("else if (fabsf(v) > amax)\n              amax = fabsf(v);",
                    "else if (v > amax)\n              amax = v;", FP8),
    "scale_constant": ("s = amax / 448.0f;", "s = amax / 447.0f;", FP8),
    "bf16_ties_away": ("(dropped == 0x8000u && (kept & 1u))", "(dropped == 0x8000u)", FP8),
    "short_copy": ("(size_t)f[d].len);", "(size_t)f[d].len - 1);", MOVES),
    "gather_stride": ("regions[r] + (int64_t)ids[i] * block_stride;\n      uint8_t* to = out",
                      "regions[r] + (int64_t)ids[i] * block_bytes;\n      uint8_t* to = out", MOVES),
    "digest_weight": ("s2 += (i + 1) * (uint64_t)p[i];", "s2 += i * (uint64_t)p[i];", MOVES),
    "scale_grid_transposed": ("scales[ti * scale_ld + tj] = s;", "scales[tj * tile_rows + ti] = s;", FP8),
    "nonfinite_code": ("q[r * q_ld + c] = 0x7F;", "q[r * q_ld + c] = 0x7E;", FP8),
    "inverse_scale_transposed": ("float s = scales[(r / 128) * scale_ld + c / 128];",
                                 "float s = scales[(c / 128) * ((rows + 127) / 128) + r / 128];", FP8),
}


def _run_pins(name, lib, suite):
    env = dict(os.environ, TC_ORACLE_LIB=lib, OMP_NUM_THREADS="2")
    r = subprocess.run([sys.executable, "-m", "pytest", suite, "-x", "-q", "-m", "not gpu",
                        "-p", "no:cacheprovider"], cwd=ROOT, env=env, capture_output=True, text=True,
                       timeout=600)
    return name, r.returncode, r.stdout[-2000:]


def test_every_mutant_fails_a_pin(tmp_path):
    src = open(os.path.join(ROOT, "oracle", "oracle.c")).read()
    jobs = []
    for name, (old, new, suite) in MUTANTS.items():
        assert src.count(old) == 1, f"mutation point of {name} not found once"
        c_path = tmp_path / f"{name}.c"
        c_path.write_text(src.replace(old, new))
        lib = str(tmp_path / f"lib{name}.so")
        oracle_build.compile_source(str(c_path), lib)
        jobs.append((name, lib, suite))
    with cf.ThreadPoolExecutor(max_workers=4) as ex:
        results = list(ex.map(lambda j: _run_pins(*j), jobs))
    survivors = [(n, out) for n, rc, out in results if rc != 1]   # 1: some test failed
    assert not survivors, "mutants not caught (or errors): " + "; ".join(
        f"{n}: {out.strip().splitlines()[-1] if out.strip() else 'no output'}" for n, out in survivors)


def test_unmutated_oracle_passes_the_same_way(tmp_path):
    """The harness itself: the unchanged source, built the same way, passes."""
    lib = str(tmp_path / "libsame.so")
    oracle_build.compile_source(os.path.join(ROOT, "oracle", "oracle.c"), lib)
    name, rc, out = _run_pins("same", lib, MOVES)
    assert rc == 0, out
