"""The device-checked build (libssm_debug.so: SSM_DEBUG, every kernel asserts
the invariants that host validation promises: positions inside the
sequence, row counts within the capacity, ids inside the vocabulary, k <= 8)
runs a tiny float32 generation and LLaDA-shaped bfloat16 steps (block start,
cached, and a batch of prompts of different lengths) without a failed check,
and gives the same outputs as the release library, bit for bit (the checks
change no arithmetic)."""
import os
import subprocess
import sys

import numpy as np
import pytest

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
DEBUG_LIB = os.path.join(ROOT, "paper_2608_23167_amd", "libssm_debug.so")


def test_debug_build_matches_release(gpu, tmp_path):
    assert os.path.exists(DEBUG_LIB), "libssm_debug.so is missing: run __graft_entry__.build()"
    out = tmp_path / "debug.npz"
    print(f"[debug build] child process with {DEBUG_LIB}", flush=True)
    r = subprocess.run([sys.executable, os.path.join(ROOT, "tests", "_debug_child.py"), DEBUG_LIB,
                        str(out)], capture_output=True, text=True, timeout=300, cwd=ROOT)
    assert r.returncode == 0, r.stdout[-2000:] + r.stderr[-4000:]
    sys.path.insert(0, os.path.join(ROOT, "tests"))
    from _debug_child import run_cases
    release = run_cases()
    debug = np.load(out)
    assert set(debug.files) == set(release)
    for key, ref in release.items():
        assert np.array_equal(debug[key], ref), key
