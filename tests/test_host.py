"""Host-side behaviour that needs no GPU: the binding refuses to work without its shared
library (no fallback path exists), bench.py refuses more than one GPU with a message, and the
entry points the build and smoke checks call exist."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_binding_fails_loudly_without_the_library(tmp_path):
    code = (
        "import sys; sys.path.insert(0, %r)\n"
        "from paper_2607_05272_amd import _lib\n"
        "_lib.LIB_PATH = %r\n"
        "_lib._lib = None\n"
        "try:\n"
        "    _lib.load()\n"
        "except ImportError as e:\n"
        "    print('raised', e)\n"
        "    sys.exit(0)\n"
        "sys.exit(3)\n" % (ROOT, str(tmp_path / "missing.so")))
    r = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "not built" in r.stdout


def test_bench_refuses_several_gpus():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr


def test_graft_entry_points_exist():
    sys.path.insert(0, ROOT)
    import __graft_entry__ as g
    assert callable(g.build) and callable(g.smoke)
