"""The oracle's pins under ASan + UBSan, and the C-ABI checks against a build
of the library whose host code carries ASan (tests/sanitize.py): both clean."""
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))


def test_host_sanitizer_runs_are_clean():
    r = subprocess.run([sys.executable, os.path.join(HERE, "sanitize.py")],
                       capture_output=True, text=True, timeout=900)
    assert r.returncode == 0, r.stdout[-4000:] + r.stderr[-4000:]
    assert "oracle pins passed" in r.stdout
    assert " passed" in r.stdout.split("library host code")[1]
