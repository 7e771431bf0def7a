"""Write the regression fixtures in this folder.  Inputs come from the seeded
generators; every expected value is computed by the CPU oracle alone.

    python tests/golden/make_golden.py
"""
import json
import os
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

import synth  # noqa: E402
from oracle import oracle as O  # noqa: E402

HERE = os.path.dirname(os.path.abspath(__file__))


def _hex(a):
    return np.ascontiguousarray(a).tobytes().hex()


def tiny_case(name, seed, M, K, N, g, with_P=True):
    c = synth.small_case(seed, M, K, N, g=g)
    dm, du = synth.default_band(K)
    P = c["P"] if with_P else None
    tM = c.get("tac_M") if g else None
    td = c.get("tac_d") if g else None
    Aq, s_a = O.quant_act(c["X"], c["state"], P, dm, du, tM, td, g)
    if with_P:
        Wq, s_w = O.prepare_weights(c["W"], P)
    else:
        Wq, s_w = O.quant_rows(c["W"].astype(np.float32))[:2]
    Y, acc = O.gemm(Aq, s_a, Wq, s_w)
    doc = {
        "name": name,
        "cites": "Eq. 9-13 (SGAT linear), Eq. 17 / App. C (TAC), Eq. 2 symmetric int4",
        "written_by": "tests/golden/make_golden.py (oracle only)",
        "M": M, "K": K, "N": N, "g": g, "dm": dm, "du": du, "has_P": with_P,
        "inputs": {"X_f16": _hex(c["X"]), "state_u8": _hex(c["state"]), "W_f16": _hex(c["W"]),
                   "P_f32": _hex(c["P"]) if with_P else None,
                   "tacM_f16": _hex(tM) if g else None, "tacd_f16": _hex(td) if g else None},
        "outputs": {"Aq_u8": _hex(Aq), "s_a_f32": _hex(s_a), "Wq_u8": _hex(Wq), "s_w_f32": _hex(s_w),
                    "acc_i32": _hex(acc), "Y_f16": _hex(Y)},
    }
    with open(os.path.join(HERE, name + ".json"), "w") as f:
        json.dump(doc, f, indent=1)
        f.write("\n")


if __name__ == "__main__":
    tiny_case("tiny_sgat_tac", 31, 8, 64, 8, 16, with_P=True)
    tiny_case("tiny_rtn", 32, 6, 64, 8, 0, with_P=False)
    print("ok")
