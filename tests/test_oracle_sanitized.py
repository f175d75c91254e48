"""The oracle under AddressSanitizer and UndefinedBehaviorSanitizer, on the CPU.

The oracle's C source is compiled with -fsanitize=address,undefined (every undefined-behaviour
report fatal) and the whole pin suite runs against that build in a subprocess, through the same
WNW_ORACLE_LIB switch the mutation tests use.  An out-of-bounds access, a use after free, a
signed overflow or a misaligned load anywhere the pins reach fails the test.  Leak detection is
off: the interpreter itself holds memory until exit.
"""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "wnw_oracle.c")


def _runtime(name):
    p = subprocess.run(["gcc", f"-print-file-name={name}"], capture_output=True, text=True).stdout.strip()
    return p if os.path.isabs(p) and os.path.exists(p) else None


def test_oracle_pins_under_asan_ubsan(tmp_path):
    asan = _runtime("libasan.so")
    if asan is None:
        pytest.skip("gcc's AddressSanitizer runtime is not installed")
    lib = str(tmp_path / "libwnw_oracle_san.so")
    cmd = ["gcc", "-O1", "-g", "-std=c99", "-fopenmp", "-fPIC", "-shared", "-Wall", "-Wextra",
           "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined", "-fno-omit-frame-pointer",
           "-o", lib, SRC, "-lm"]
    subprocess.run(cmd, check=True)
    env = dict(os.environ)
    env["WNW_ORACLE_LIB"] = lib
    # the sanitizer runtime must come first among the preloaded libraries of the interpreter;
    # whatever the environment already preloads stays after it
    env["LD_PRELOAD"] = ":".join(x for x in (asan, env.get("LD_PRELOAD", "")) if x)
    # reports go to files: a sanitizer that ends the interpreter inside a test would otherwise
    # take pytest's captured output with it
    logs = tmp_path / "san"
    env["ASAN_OPTIONS"] = f"detect_leaks=0:verify_asan_link_order=0:log_path={logs}"
    env["UBSAN_OPTIONS"] = f"halt_on_error=1:print_stacktrace=1:log_path={logs}"
    env["OMP_NUM_THREADS"] = "4"
    r = subprocess.run([sys.executable, "-m", "pytest", os.path.join(ROOT, "tests", "test_oracle_pins.py"), "-x", "-q",
                        "-p", "no:cacheprovider"], cwd=ROOT, env=env, capture_output=True, text=True, timeout=1200)
    out = r.stdout + r.stderr
    reports = "".join(open(tmp_path / f).read() for f in os.listdir(tmp_path) if f.startswith("san"))
    assert r.returncode == 0 and not reports, (reports + out)[-4000:]
    assert " passed" in out


def test_sanitizer_catches_a_planted_overflow(tmp_path):
    """The same build and run catch a heap overflow planted in a copy of the oracle (so the
    sanitized library is the one the pins load)."""
    asan = _runtime("libasan.so")
    if asan is None:
        pytest.skip("gcc's AddressSanitizer runtime is not installed")
    src = open(SRC).read()
    anchor = "    for (int32_t j = 0; j < d; ++j) out[j] = 0.0;\n    if (n == 0) return;\n"
    assert anchor in src
    planted = src.replace(anchor, anchor + "    { double *t_ = malloc(2 * sizeof(double)); ((volatile double *)t_)[2] = 1.0; free(t_); }\n", 1)
    if "#include <stdlib.h>" not in planted:
        planted = "#include <stdlib.h>\n" + planted
    msrc = tmp_path / "planted.c"
    msrc.write_text(planted)
    lib = str(tmp_path / "libplanted.so")
    subprocess.run(["gcc", "-O1", "-g", "-std=c99", "-fopenmp", "-fPIC", "-shared", "-fsanitize=address,undefined",
                    "-fno-omit-frame-pointer", "-I", os.path.dirname(SRC), "-o", lib, str(msrc), "-lm"], check=True)
    env = dict(os.environ)
    env["WNW_ORACLE_LIB"] = lib
    env["LD_PRELOAD"] = ":".join(x for x in (asan, env.get("LD_PRELOAD", "")) if x)
    env["ASAN_OPTIONS"] = "detect_leaks=0:verify_asan_link_order=0"
    env["OMP_NUM_THREADS"] = "1"
    # -s: the report reaches this process's pipes even though the sanitizer ends the interpreter
    r = subprocess.run([sys.executable, "-m", "pytest", os.path.join(ROOT, "tests", "test_oracle_pins.py"), "-x", "-q",
                        "-s", "-p", "no:cacheprovider", "-k", "full_budget"], cwd=ROOT, env=env, capture_output=True,
                       text=True, timeout=600)
    assert r.returncode != 0
    assert "heap-buffer-overflow" in r.stdout + r.stderr
