"""The C-ABI argument checks (tests/test_abi.py) once more against a copy of
the library whose C-ABI layer is built with AddressSanitizer and
UndefinedBehaviorSanitizer on the host: an invalid read or write, a
misaligned or out-of-range load or an overflow in the descriptor checks and
workspace planning ends the run with a report.  CPU only."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_abi_checks_under_host_sanitizers(tmp_path):
    sys.path.insert(0, ROOT)
    from paper_1910_13444_amd import build_sanitized as bs
    try:
        rt = bs.asan_runtime()
    except RuntimeError as e:
        pytest.skip(str(e))
    lib = bs.build_sanitized(jobs=4)
    log = tmp_path / "san"
    env = dict(os.environ, LD_PRELOAD=rt, PIGAN_LIBRARY=lib,
               ASAN_OPTIONS=f"detect_leaks=0:halt_on_error=1:log_path={log}",
               UBSAN_OPTIONS=f"halt_on_error=1:print_stacktrace=1:log_path={log}")
    r = subprocess.run([sys.executable, "-m", "pytest", os.path.join(ROOT, "tests", "test_abi.py"), "-q",
                        "-p", "no:cacheprovider"], env=env, cwd=ROOT, capture_output=True, text=True, timeout=600)
    reports = "".join(p.read_text() for p in tmp_path.glob("san*"))
    assert r.returncode == 0 and not reports, (r.stdout[-3000:] + r.stderr[-3000:] + reports[:4000])
    assert " passed" in r.stdout
