"""Helpers for the GPU parity tests: numpy <-> device copies and comparisons."""
import sys

import numpy as np
import torch


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def dev(a):
    if a is None:
        return None
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def host(t):
    torch.cuda.synchronize()
    return t.cpu().numpy()


def assert_bits(got, ref, what):
    got = np.ascontiguousarray(got)
    ref = np.ascontiguousarray(ref)
    assert got.shape == ref.shape, (what, got.shape, ref.shape)
    if got.tobytes() != ref.tobytes():
        g = got.view(np.uint8).reshape(got.shape[0], -1) if got.ndim else got
        r = ref.view(np.uint8).reshape(ref.shape[0], -1) if ref.ndim else ref
        bad = np.argwhere(g != r)
        raise AssertionError(f"{what}: {len(bad)} differing bytes, first at {bad[:5].tolist()}")


# fp16 outputs: within 1e-3 relative / 1e-2 absolute of the oracle (the stated
# tolerance), and in fact bit-identical because the arithmetic order is fixed.
Y_RTOL, Y_ATOL = 1e-3, 1e-2


def assert_y(got, ref, what="Y"):
    g = got.astype(np.float64)
    r = ref.astype(np.float64)
    assert np.all(np.abs(g - r) <= Y_ATOL + Y_RTOL * np.abs(r)), what + ": outside tolerance"
    assert_bits(got, ref, what)


def pack_codes(q):
    q = np.asarray(q, np.int64)
    return ((q[:, 0::2] & 15) | ((q[:, 1::2] & 15) << 4)).astype(np.uint8)
