"""The C oracle built with AddressSanitizer and UndefinedBehaviorSanitizer
runs the whole pin battery (tests/test_oracle_pins.py) without a report:
no out-of-bounds access, use after free, signed overflow, misaligned load
or other undefined behaviour in any pinned case (CPU only).  A negative
control plants a one-past-the-end read in a copy of the oracle and checks
that the same run then fails."""
import os
import subprocess
import sys

import oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SAN_FLAGS = ("-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
             "-fno-sanitize-recover=all")


def _sanitized_pins(tmp_path, src=None, select=None):
    so = str(tmp_path / "libdopr_oracle_san.so")
    oracle.build(**({"src": src} if src else {}), out=so,
                 extra_flags=SAN_FLAGS)
    r = subprocess.run(["gcc", "-print-file-name=libasan.so"],
                       capture_output=True, text=True, check=True)
    asan = r.stdout.strip()
    assert os.path.isabs(asan), "gcc has no AddressSanitizer runtime"
    env = dict(os.environ)
    env.update(DOPR_ORACLE_LIB=so,
               LD_PRELOAD=asan,   # the interpreter itself is not instrumented
               ASAN_OPTIONS="detect_leaks=0:exitcode=97",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1:exitcode=98",
               PYTHONDONTWRITEBYTECODE="1")
    # -s: a sanitizer report goes straight to stderr, not to pytest's capture
    cmd = [sys.executable, "-m", "pytest", "-x", "-q", "-s", "-p",
           "no:cacheprovider",
           os.path.join(ROOT, "tests", "test_oracle_pins.py")]
    if select:
        cmd += ["-k", select]
    return subprocess.run(cmd, env=env, cwd=ROOT, capture_output=True,
                          text=True, timeout=1200)


def test_oracle_pins_under_asan_and_ubsan(tmp_path):
    r = _sanitized_pins(tmp_path)
    tail = r.stdout[-4000:] + "\n" + r.stderr[-4000:]
    assert r.returncode == 0, tail
    assert "AddressSanitizer" not in r.stderr, tail
    assert "runtime error" not in r.stderr, tail
    assert " passed" in r.stdout, tail


def test_sanitized_run_catches_a_planted_overread(tmp_path):
    src = open(os.path.join(ROOT, "oracle", "dopr_oracle.c")).read()
    loop = ("    for (int i = 0; i < width; ++i) {\n"
            "      ly += wy[i] * hh[i];")
    assert src.count(loop) == 1
    bad = tmp_path / "overread.c"
    bad.write_text(src.replace(loop, loop.replace("i < width", "i <= width")))
    r = _sanitized_pins(tmp_path, src=str(bad), select="pin_score")
    assert r.returncode == 97, r.stderr[-3000:]     # ASan's exit code
    assert "heap-buffer-overflow" in r.stderr, r.stderr[-3000:]
