"""The binding imported before anything else in a fresh process: it brings in
torch's HIP runtime before the library binds to one, so a search runs (a
second copy of the runtime would fail the first launch)."""
import os
import subprocess
import sys

import pytest

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

SCRIPT = """
import sys
sys.path.insert(0, {root!r})
from paper_2609_02109_amd import mf, synth
inst = synth.cfg0(0)
r = mf.Problem(inst).search(inst.sla, inst.omega, k=1)
print("found", int(r["n_feas"]), flush=True)
"""


def test_binding_first_in_a_fresh_process():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    r = subprocess.run([sys.executable, "-c", SCRIPT.format(root=ROOT)], capture_output=True, text=True,
                       timeout=300)
    assert r.returncode == 0, r.stderr[-2000:]
    assert "found" in r.stdout
