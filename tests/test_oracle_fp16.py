"""Pins of the oracle's IEEE binary16 conversions against numpy's (an independent
implementation of the same IEEE 754 definition: exact widening, RNE narrowing)."""
import numpy as np

from oracle import oracle as O


def test_h2f_exhaustive():
    h = np.arange(65536, dtype=np.uint16)
    got = O.h2f(h)
    ref = h.view(np.float16).astype(np.float32)
    same = (got.view(np.uint32) == ref.view(np.uint32)) | (np.isnan(got) & np.isnan(ref))
    assert same.all()


def test_f2h_roundtrip_exhaustive():
    h = np.arange(65536, dtype=np.uint16)
    f = h.view(np.float16).astype(np.float32)
    finite = np.isfinite(f)
    back = O.f2h(f[finite])
    assert (back == h[finite]).all()


def _check_against_numpy(f):
    f = np.asarray(f, np.float32)
    got = O.f2h(f)
    ref = f.astype(np.float16).view(np.uint16)
    bad = np.nonzero(got != ref)[0]
    assert len(bad) == 0, (f[bad[:5]], got[bad[:5]], ref[bad[:5]])


def test_f2h_midpoints_and_neighbours():
    # every midpoint between consecutive finite positive halves, and one fp32 ulp around it
    h = np.arange(0, 0x7BFF, dtype=np.uint16)
    lo = h.view(np.float16).astype(np.float64)
    hi = (h + 1).view(np.float16).astype(np.float64)
    mid = ((lo + hi) / 2).astype(np.float32)       # exact in fp32 (<= 12 significant bits)
    assert (mid.astype(np.float64) == (lo + hi) / 2).all()
    for v in (mid, np.nextafter(mid, np.float32(0)), np.nextafter(mid, np.float32(np.inf))):
        _check_against_numpy(v)
        _check_against_numpy(-v)


def test_f2h_ranges():
    rng = np.random.default_rng(5)
    e = rng.uniform(-30, 17, 200000)
    v = (rng.uniform(1, 2, e.size) * 2.0 ** e).astype(np.float32)
    _check_against_numpy(v)
    _check_against_numpy(-v)
    edges = np.array([0.0, -0.0, 65504.0, 65519.996, 65520.0, 65536.0, 1e30, np.inf,
                      2.0 ** -24, 2.0 ** -25, 2.0 ** -25 * 1.0000001, 2.0 ** -26, 2.0 ** -14,
                      2.0 ** -14 - 2.0 ** -25, 1e-45], np.float32)
    _check_against_numpy(edges)
    _check_against_numpy(-edges)
