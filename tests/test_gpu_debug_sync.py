"""SQ_DEBUG_SYNC: with the switch set, every launch is followed by a device
synchronisation and an error check; results are unchanged.  Run in a child
process so that the library reads the variable afresh."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

CHILD = r"""
import numpy as np, torch, sys
sys.path.insert(0, ROOT)
import paper_2606_04945_amd as sq, synth
from oracle import oracle as O
c = synth.small_case(3, 40, 256, 24, g=16)
dm, du = synth.default_band(256)
T = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
Wq, s_w = sq.sgat_prepare_weights(T(c["W"]), T(c["P"]))
Aq, s_a = sq.sgat_quant_act(T(c["X"]), T(c["state"]), T(c["P"]), dm, du, T(c["tac_M"]), T(c["tac_d"]), 16)
Y, acc = sq.w4a4_gemm(Aq, s_a, Wq, s_w, want_acc=True)
torch.cuda.synchronize()
ref = O.sgat_linear(c["X"], c["state"], c["P"], c["W"], dm, du, c["tac_M"], c["tac_d"], 16)
assert acc.cpu().numpy().tobytes() == np.ascontiguousarray(ref["acc"]).tobytes()
assert Y.cpu().numpy().tobytes() == np.ascontiguousarray(ref["Y"]).tobytes()
print("ok", flush=True)
""".replace("ROOT", repr(ROOT))


@pytest.mark.gpu
def test_debug_sync_switch_leaves_results_unchanged():
    env = dict(os.environ, SQ_DEBUG_SYNC="1")
    r = subprocess.run([sys.executable, "-c", CHILD], capture_output=True, text=True, env=env, timeout=300)
    assert r.returncode == 0 and r.stdout.strip().endswith("ok"), r.stderr[-2000:]
