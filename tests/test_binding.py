"""The binding has no fallback: without the built HIP library every entry
point fails loudly (checked in a fresh interpreter, since a loaded library is
cached per process)."""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_missing_library_raises():
    code = ("from paper_2603_00188_amd import stlite as S\n"
            "try:\n"
            "    S.load('/nonexistent/libstlite.so')\n"
            "except RuntimeError as e:\n"
            "    print('raised:', e)\n"
            "    raise SystemExit(3)\n")
    r = subprocess.run([sys.executable, "-c", code], cwd=ROOT, capture_output=True, text=True, timeout=120)
    assert r.returncode == 3, r.stdout + r.stderr
    assert "is missing" in r.stdout
