"""The oracle reproduces its committed regression fixtures bit for bit."""
import glob
import json
import os

import numpy as np
import pytest

from oracle import oracle as O

GOLD = sorted(glob.glob(os.path.join(os.path.dirname(__file__), "golden", "*.json")))


def load(path):
    with open(path) as f:
        d = json.load(f)
    M, K, N = d["M"], d["K"], d["N"]
    i, o = d["inputs"], d["outputs"]

    def arr(hx, dt, shape):
        return None if hx is None else np.frombuffer(bytes.fromhex(hx), dt).reshape(shape).copy()
    g = d["g"]
    ins = dict(X=arr(i["X_f16"], np.float16, (M, K)), state=arr(i["state_u8"], np.uint8, (M,)),
               W=arr(i["W_f16"], np.float16, (N, K)), P=arr(i["P_f32"], np.float32, (K, K)),
               tac_M=arr(i["tacM_f16"], np.float16, (K // g, g, g)) if g else None,
               tac_d=arr(i["tacd_f16"], np.float16, (K,)) if g else None)
    outs = dict(Aq=arr(o["Aq_u8"], np.uint8, (M, K // 2)), s_a=arr(o["s_a_f32"], np.float32, (M,)),
                Wq=arr(o["Wq_u8"], np.uint8, (N, K // 2)), s_w=arr(o["s_w_f32"], np.float32, (N,)),
                acc=arr(o["acc_i32"], np.int32, (M, N)), Y=arr(o["Y_f16"], np.float16, (M, N)))
    return d, ins, outs


@pytest.mark.parametrize("path", GOLD, ids=[os.path.basename(p) for p in GOLD])
def test_golden(path):
    d, ins, outs = load(path)
    Aq, s_a = O.quant_act(ins["X"], ins["state"], ins["P"], d["dm"], d["du"],
                          ins["tac_M"], ins["tac_d"], d["g"])
    if d["has_P"]:
        Wq, s_w = O.prepare_weights(ins["W"], ins["P"])
    else:
        Wq, s_w = O.quant_rows(ins["W"].astype(np.float32))[:2]
    Y, acc = O.gemm(Aq, s_a, Wq, s_w)
    for k, v in dict(Aq=Aq, s_a=s_a, Wq=Wq, s_w=s_w, acc=acc, Y=Y).items():
        assert v.tobytes() == outs[k].tobytes(), k
