"""Host-side checks of the C ABI (no GPU needed): the library loads, exports every
function include/starquant.h declares, and rejects bad arguments before touching
the device."""
import ctypes
import os
import re

import pytest

from paper_2606_04945_amd import _lib as L

HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include", "starquant.h")


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?[a-z_0-9]+\s*\*?\s*([a-z_0-9]+)\s*\(", src, flags=re.M)))


@pytest.fixture(scope="module")
def lib():
    return L.lib()


def test_exports_every_declared_function(lib):
    names = declared_functions()
    assert {"sgat_prepare_weights", "sgat_quant_act", "w4a4_gemm", "tac_apply"} <= set(names)
    for n in names:
        assert hasattr(lib, n), n
        assert n in L.SIGNATURES, n


def test_helpers(lib):
    assert lib.sq_version().startswith(b"starquant")
    assert lib.sq_tac_default_block(4096) == 16
    assert lib.sq_tac_default_block(3584) == 16
    assert lib.sq_tac_default_block(360) == 15
    assert lib.sq_tac_default_block(17) == 1
    assert lib.sq_tac_default_block(0) == 0
    assert lib.sq_quant_act_workspace_bytes(0, 4096, 1, 1) == 0
    assert lib.sq_quant_act_workspace_bytes(1024, 4096, 0, 0) == 0
    assert lib.sq_quant_act_workspace_bytes(1024, 4096, 1, 0) == 1024 * 4096 * 4
    assert lib.sq_quant_act_workspace_bytes(1024, 4096, 1, 1) == 1024 * 4096 * 6
    assert lib.sq_prepare_weights_workspace_bytes(64, 512, 1) == 64 * 512 * 4
    assert lib.sq_prepare_weights_workspace_bytes(64, 512, 0) == 0
    assert lib.sq_gemm_workspace_bytes(4096, 4096, 4096) == 0      # no split at large M
    assert lib.sq_gemm_workspace_bytes(96, 4096, 12288) > 0        # split-K across workgroups: few tiles, long K
    assert lib.sq_gemm_workspace_bytes(48, 4096, 12288) == 0       # M <= 48 splits K inside the workgroup


FAKE = 1 << 20          # a 16-byte aligned non-null address; never dereferenced on these paths


@pytest.mark.parametrize("K", [0, 32, 100, 130, 131072 + 64])
def test_bad_K_rejected(lib, K):
    assert lib.sgat_quant_act(FAKE, FAKE, FAKE, 4, K, 0, 0, None, None, 0, FAKE, FAKE, FAKE, 1 << 30, None) \
        == L.SQ_ERR_SHAPE
    assert lib.w4a4_gemm(FAKE, FAKE, FAKE, FAKE, 4, 16, K, FAKE, None, FAKE, 1 << 30, None) == L.SQ_ERR_SHAPE
    assert b"K=" in lib.sq_last_error()


def test_bad_bands_and_tac_rejected(lib):
    assert lib.sgat_quant_act(FAKE, FAKE, None, 4, 64, 32, 32, None, None, 0, FAKE, FAKE, None, 0, None) \
        == L.SQ_ERR_SHAPE
    assert lib.sgat_quant_act(FAKE, FAKE, None, 4, 64, -1, 0, None, None, 0, FAKE, FAKE, None, 0, None) \
        == L.SQ_ERR_SHAPE
    for g in (0, 3, 256, 48):
        assert lib.sgat_quant_act(FAKE, FAKE, None, 4, 128, 4, 4, FAKE, FAKE, g, FAKE, FAKE, FAKE, 1 << 30, None) \
            == L.SQ_ERR_SHAPE
        assert lib.tac_apply(FAKE, FAKE, FAKE, 4, 128, g, FAKE + (1 << 16), None) == L.SQ_ERR_SHAPE
    # tac_M without tac_d
    assert lib.sgat_quant_act(FAKE, FAKE, None, 4, 128, 4, 4, FAKE, None, 16, FAKE, FAKE, FAKE, 1 << 30, None) \
        == L.SQ_ERR_NULL


def test_null_alignment_workspace(lib):
    assert lib.sgat_quant_act(None, None, None, 4, 64, 2, 2, None, None, 0, FAKE, FAKE, None, 0, None) \
        == L.SQ_ERR_NULL
    assert lib.sgat_quant_act(FAKE + 2, None, None, 4, 64, 2, 2, None, None, 0, FAKE, FAKE, None, 0, None) \
        == L.SQ_ERR_ALIGN
    need = lib.sq_quant_act_workspace_bytes(4, 64, 1, 0)
    assert lib.sgat_quant_act(FAKE, None, FAKE, 4, 64, 2, 2, None, None, 0, FAKE, FAKE, FAKE, need - 1, None) \
        == L.SQ_ERR_WORKSPACE
    assert lib.sgat_quant_act(FAKE, None, FAKE, 4, 64, 2, 2, None, None, 0, FAKE, FAKE, None, need, None) \
        == L.SQ_ERR_WORKSPACE
    assert lib.w4a4_gemm(FAKE, FAKE, FAKE, FAKE, 4, 12, 64, FAKE, None, None, 0, None) == L.SQ_ERR_SHAPE   # N % 8
    assert lib.w4a4_gemm(FAKE, FAKE, FAKE, FAKE, 4, 16, 64, None, None, None, 0, None) == L.SQ_ERR_NULL
    wneed = lib.sq_gemm_workspace_bytes(96, 4096, 12288)
    assert lib.w4a4_gemm(FAKE, FAKE, FAKE, FAKE, 96, 4096, 12288, FAKE, None, None, 0, None) == L.SQ_ERR_WORKSPACE
    assert wneed > 0
    assert lib.sgat_prepare_weights(FAKE, FAKE, 8, 64, FAKE, FAKE, None, 0, None) == L.SQ_ERR_WORKSPACE
    assert lib.sgat_transform(FAKE, None, FAKE + 4, 8, 64, 0, 0, FAKE, None) == L.SQ_ERR_ALIGN
    assert lib.sgat_quantize(None, 8, 64, FAKE, FAKE, None) == L.SQ_ERR_NULL
    # overlapping TAC output
    assert lib.tac_apply(FAKE, FAKE, FAKE, 4, 128, 16, FAKE + 256, None) == L.SQ_ERR_SHAPE


def test_empty_is_a_no_op(lib):
    # M == 0 returns success without any device work (and without a device)
    assert lib.sgat_quant_act(None, None, None, 0, 64, 2, 2, None, None, 0, None, None, None, 0, None) == L.SQ_OK
    assert lib.w4a4_gemm(None, None, None, None, 0, 16, 64, None, None, None, 0, None) == L.SQ_OK
    assert lib.w4a4_gemm(None, None, None, None, 4, 0, 64, None, None, None, 0, None) == L.SQ_OK
    assert lib.tac_apply(None, None, None, 0, 64, 16, None, None) == L.SQ_OK
    assert lib.sgat_prepare_weights(None, None, 0, 64, None, None, None, 0, None) == L.SQ_OK
    assert lib.sgat_transform(None, None, None, 0, 64, 0, 0, None, None) == L.SQ_OK
    assert lib.sgat_quantize(None, 0, 64, None, None, None) == L.SQ_OK


def test_binding_fails_loudly_without_library(monkeypatch, tmp_path):
    import importlib
    monkeypatch.setattr(L, "LIB_PATH", str(tmp_path / "missing.so"))
    monkeypatch.setattr(L, "_lib", None)
    with pytest.raises(ImportError):
        L.lib()
    importlib.reload(L)


def test_w8_entry_points_validate(lib):
    assert lib.w8a8_gemm(FAKE, FAKE, FAKE, FAKE, 4, 16, 65536 + 64, FAKE, None, FAKE, 1 << 30, None) == L.SQ_ERR_SHAPE
    assert b"65536" in lib.sq_last_error()
    assert lib.w8a8_gemm(None, None, None, None, 0, 16, 64, None, None, None, 0, None) == L.SQ_OK
    assert lib.sgat_quant_act_w8(FAKE, None, None, 4, 100, 0, 0, None, None, 0, FAKE, FAKE, None, 0, None) \
        == L.SQ_ERR_SHAPE
    assert lib.sgat_quantize_w8(None, 4, 64, FAKE, FAKE, None) == L.SQ_ERR_NULL
    assert lib.sgat_prepare_weights_w8(FAKE, FAKE, 8, 64, FAKE, FAKE, None, 0, None) == L.SQ_ERR_WORKSPACE
    assert lib.sq_gemm_w8_workspace_bytes(4096, 4096, 4096) == 0
    # operands of 2 GiB or more are refused (32-bit buffer offsets)
    assert lib.w4a4_gemm(FAKE, FAKE, FAKE, FAKE, 65536, 16, 65536, FAKE, None, FAKE, 1 << 40, None) == L.SQ_ERR_SHAPE


def test_row_limit_of_tiled_launches(lib):
    big = 65535 * 64 + 1
    assert lib.w4a4_gemm(FAKE, FAKE, FAKE, FAKE, big, 16, 64, FAKE, None, FAKE, 1 << 40, None) == L.SQ_ERR_SHAPE
    assert b"rows" in lib.sq_last_error()
    assert lib.tac_apply(FAKE, FAKE, FAKE, big, 64, 16, FAKE + (1 << 40), None) == L.SQ_ERR_SHAPE
    assert lib.sgat_quant_act(FAKE, FAKE, None, big, 64, 2, 2, FAKE, FAKE, 16, FAKE, FAKE, FAKE, 1 << 40, None) \
        == L.SQ_ERR_SHAPE


def test_tac_calibrate_validates(lib):
    assert lib.sq_tac_calibrate_workspace_bytes(1000, 4096, 16) > 0
    assert lib.sq_tac_calibrate_workspace_bytes(0, 4096, 16) == 0
    ok = (3e-4, 1e-8, 0.15, 0.55)
    big = 1 << 40
    assert lib.tac_calibrate(FAKE, FAKE, 0, 64, 16, *ok, FAKE, FAKE, None, None, FAKE, big, None) == L.SQ_ERR_SHAPE
    assert lib.tac_calibrate(FAKE, FAKE, 8, 64, 3, *ok, FAKE, FAKE, None, None, FAKE, big, None) == L.SQ_ERR_SHAPE
    assert lib.tac_calibrate(FAKE, FAKE, 8, 100, 4, *ok, FAKE, FAKE, None, None, FAKE, big, None) == L.SQ_ERR_SHAPE
    assert lib.tac_calibrate(FAKE, FAKE, 8, 64, 16, 3e-4, 1e-8, 1.5, 0.55, FAKE, FAKE, None, None, FAKE, big, None) \
        == L.SQ_ERR_SHAPE
    assert lib.tac_calibrate(FAKE, FAKE, 8, 64, 16, -1.0, 1e-8, 0.1, 0.5, FAKE, FAKE, None, None, FAKE, big, None) \
        == L.SQ_ERR_SHAPE
    assert lib.tac_calibrate(FAKE, None, 8, 64, 16, *ok, FAKE, FAKE, None, None, FAKE, big, None) == L.SQ_ERR_NULL
    assert lib.tac_calibrate(FAKE, FAKE, 8, 64, 16, *ok, FAKE, FAKE, None, None, None, big, None) == L.SQ_ERR_NULL
    assert lib.tac_calibrate(FAKE, FAKE, 8, 64, 16, *ok, FAKE + 8, FAKE, None, None, FAKE, big, None) \
        == L.SQ_ERR_ALIGN
    need = lib.sq_tac_calibrate_workspace_bytes(8, 64, 16)
    assert lib.tac_calibrate(FAKE, FAKE, 8, 64, 16, *ok, FAKE, FAKE, None, None, FAKE, need - 1, None) \
        == L.SQ_ERR_WORKSPACE


def test_fp6_entry_points_validate(lib):
    assert lib.sq_fp6_row_bytes(64) == 96 and lib.sq_fp6_row_bytes(128) == 96
    assert lib.sq_fp6_row_bytes(3584) == 96 * 28 and lib.sq_fp6_row_bytes(4160) == 96 * 33
    assert lib.sq_fp6_row_bytes(100) == 0 and lib.sq_fp6_row_bytes(0) == 0
    # K, N % 8, NULL, alignment
    assert lib.w4a4_gemm_fp6(FAKE, FAKE, FAKE, FAKE, 4, 16, 100, FAKE, None, None) == L.SQ_ERR_SHAPE
    assert lib.w4a4_gemm_fp6(FAKE, FAKE, FAKE, FAKE, 4, 12, 128, FAKE, None, None) == L.SQ_ERR_SHAPE
    assert lib.w4a4_gemm_fp6(FAKE, FAKE, FAKE, FAKE, 4, 16, 128, None, None, None) == L.SQ_ERR_NULL
    assert lib.w4a4_gemm_fp6(FAKE + 8, FAKE, FAKE, FAKE, 4, 16, 128, FAKE, None, None) == L.SQ_ERR_ALIGN
    assert lib.w4a4_gemm_fp6(None, None, None, None, 0, 16, 128, None, None, None) == L.SQ_OK
    # operands over 2 GiB
    assert lib.w4a4_gemm_fp6(FAKE, FAKE, FAKE, FAKE, 1 << 20, 16, 4096, FAKE, None, None) == L.SQ_ERR_SHAPE
    # conversion: K, NULL, alignment, overlap
    assert lib.sq_codes_to_fp6(FAKE, 4, 96, FAKE + (1 << 20), None) == L.SQ_ERR_SHAPE
    assert lib.sq_codes_to_fp6(None, 4, 128, FAKE, None) == L.SQ_ERR_NULL
    assert lib.sq_codes_to_fp6(FAKE, 4, 128, FAKE + 8, None) == L.SQ_ERR_ALIGN
    assert lib.sq_codes_to_fp6(FAKE, 4, 128, FAKE + 64, None) == L.SQ_ERR_SHAPE
    assert lib.sq_codes_to_fp6(None, 0, 128, None, None) == L.SQ_OK


def test_frag_entry_points_validate(lib):
    # ceil(N / 16) ceil(K / 128) 1024
    assert lib.sq_frag_weight_bytes(16, 128) == 1024 and lib.sq_frag_weight_bytes(24, 192) == 2 * 2 * 1024
    assert lib.sq_frag_weight_bytes(24576, 4096) == 1536 * 32 * 1024 and lib.sq_frag_weight_bytes(0, 128) == 0
    assert lib.sq_frag_weight_bytes(16, 100) == 0 and lib.sq_frag_weight_bytes(-1, 128) == 0
    # GEMM: K, N % 8, NULL, alignment, workspace, empty, over 2 GiB
    args = (FAKE, FAKE, FAKE, FAKE)
    assert lib.w4a4_gemm_frag(*args, 4, 16, 100, FAKE, None, None, 0, None) == L.SQ_ERR_SHAPE
    assert lib.w4a4_gemm_frag(*args, 4, 12, 128, FAKE, None, None, 0, None) == L.SQ_ERR_SHAPE
    assert lib.w4a4_gemm_frag(*args, -1, 16, 128, FAKE, None, None, 0, None) == L.SQ_ERR_SHAPE
    assert lib.w4a4_gemm_frag(*args, 4, 16, 128, None, None, None, 0, None) == L.SQ_ERR_NULL
    assert lib.w4a4_gemm_frag(FAKE, FAKE, None, FAKE, 4, 16, 128, FAKE, None, None, 0, None) == L.SQ_ERR_NULL
    assert lib.w4a4_gemm_frag(FAKE, FAKE, FAKE + 8, FAKE, 4, 16, 128, FAKE, None, None, 0, None) == L.SQ_ERR_ALIGN
    assert lib.w4a4_gemm_frag(None, None, None, None, 0, 16, 128, None, None, None, 0, None) == L.SQ_OK
    assert lib.w4a4_gemm_frag(*args, 1 << 20, 16, 4096, FAKE, None, None, 0, None) == L.SQ_ERR_SHAPE
    assert lib.w4a4_gemm_frag(*args, 4, 1 << 20, 4096, FAKE, None, None, 0, None) == L.SQ_ERR_SHAPE
    need = lib.sq_gemm_workspace_bytes(96, 4096, 4096)
    assert need > 0
    assert lib.w4a4_gemm_frag(*args, 96, 4096, 4096, FAKE, None, None, need - 1, None) == L.SQ_ERR_WORKSPACE
    assert lib.w4a4_gemm_frag(*args, 96, 4096, 4096, FAKE, None, None, need, None) == L.SQ_ERR_WORKSPACE
    # conversion: K, N, NULL, alignment, overlap, empty, over 2 GiB
    assert lib.sq_weights_to_frag(FAKE, 16, 96, FAKE + (1 << 20), None) == L.SQ_ERR_SHAPE
    assert lib.sq_weights_to_frag(FAKE, -16, 128, FAKE + (1 << 20), None) == L.SQ_ERR_SHAPE
    assert lib.sq_weights_to_frag(None, 16, 128, FAKE, None) == L.SQ_ERR_NULL
    assert lib.sq_weights_to_frag(FAKE, 16, 128, FAKE + 8, None) == L.SQ_ERR_ALIGN
    assert lib.sq_weights_to_frag(FAKE, 16, 128, FAKE + 512, None) == L.SQ_ERR_SHAPE
    assert lib.sq_weights_to_frag(FAKE + 512, 16, 128, FAKE, None) == L.SQ_ERR_SHAPE
    assert lib.sq_weights_to_frag(None, 0, 128, None, None) == L.SQ_OK
    assert lib.sq_weights_to_frag(FAKE, 1 << 20, 4096, FAKE + (1 << 40), None) == L.SQ_ERR_SHAPE


def test_w8_frag_entry_points_validate(lib):
    # ceil(N / 16) ceil(K / 64) 1024: the bytes of 2 K int4 codes
    assert lib.sq_frag_weight_w8_bytes(16, 64) == 1024 and lib.sq_frag_weight_w8_bytes(24, 96) == 0
    assert lib.sq_frag_weight_w8_bytes(24, 192) == 2 * 3 * 1024
    assert lib.sq_frag_weight_w8_bytes(16, 65536 + 64) == 0 and lib.sq_frag_weight_w8_bytes(-1, 128) == 0
    args = (FAKE, FAKE, FAKE, FAKE)
    f = lib.w8a8_gemm_frag
    assert f(*args, 4, 16, 65536 + 64, FAKE, None, FAKE, 1 << 30, None) == L.SQ_ERR_SHAPE
    assert b"65536" in lib.sq_last_error()
    assert f(*args, 4, 12, 128, FAKE, None, None, 0, None) == L.SQ_ERR_SHAPE
    assert f(*args, 4, 16, 128, None, None, None, 0, None) == L.SQ_ERR_NULL
    assert f(FAKE, FAKE, FAKE + 8, FAKE, 4, 16, 128, FAKE, None, None, 0, None) == L.SQ_ERR_ALIGN
    assert f(None, None, None, None, 0, 16, 128, None, None, None, 0, None) == L.SQ_OK
    assert f(*args, 1 << 16, 16, 65536, FAKE, None, None, 0, None) == L.SQ_ERR_SHAPE      # 4 GiB of codes
    need = lib.sq_gemm_w8_workspace_bytes(96, 4096, 4096)
    assert need > 0
    assert f(*args, 96, 4096, 4096, FAKE, None, None, need - 1, None) == L.SQ_ERR_WORKSPACE
    assert lib.sq_weights_to_frag_w8(FAKE, 16, 65536 + 64, FAKE + (1 << 40), None) == L.SQ_ERR_SHAPE
    assert lib.sq_weights_to_frag_w8(FAKE, 16, 96, FAKE + (1 << 20), None) == L.SQ_ERR_SHAPE
    assert lib.sq_weights_to_frag_w8(None, 16, 128, FAKE, None) == L.SQ_ERR_NULL
    assert lib.sq_weights_to_frag_w8(FAKE, 16, 128, FAKE + 1024, None) == L.SQ_ERR_SHAPE   # overlap: 2 KB rows
    assert lib.sq_weights_to_frag_w8(None, 0, 128, None, None) == L.SQ_OK


def test_noalloc_gemm_validates(lib):
    args = (FAKE, FAKE, FAKE, FAKE)
    f = lib.w4a4_gemm_frag_noalloc
    assert f(*args, 4, 16, 100, FAKE, None, None) == L.SQ_ERR_SHAPE
    assert f(*args, 4, 12, 128, FAKE, None, None) == L.SQ_ERR_SHAPE
    assert f(*args, -1, 16, 128, FAKE, None, None) == L.SQ_ERR_SHAPE
    assert f(*args, 4, 16, 128, None, None, None) == L.SQ_ERR_NULL
    assert f(FAKE, FAKE, FAKE + 8, FAKE, 4, 16, 128, FAKE, None, None) == L.SQ_ERR_ALIGN
    assert f(*args, 1 << 20, 16, 4096, FAKE, None, None) == L.SQ_ERR_SHAPE
    assert f(None, None, None, None, 0, 16, 128, None, None, None) == L.SQ_OK
    assert f(None, None, None, None, 4, 0, 128, None, None, None) == L.SQ_OK


def test_noalloc_scratch_covers_every_split_shape(lib):
    """The GEMM splits K only below 256 output tiles of 64 x 64, so the partial
    sums never exceed the 16 MiB the no-allocation entry point holds: checked
    over token counts, widths and depths on both sides of every threshold."""
    cap = 16 << 20
    worst = 0
    for M in (17, 49, 64, 65, 100, 128, 200, 255, 256, 300, 512, 1000, 1024, 2048, 4096):
        for N in (8, 64, 520, 1024, 2048, 4096, 4608, 8192, 12288, 16384, 24576, 37888, 65536):
            for K in (64, 512, 4096, 8192, 12288, 18944, 65536, 131072):
                worst = max(worst, lib.sq_gemm_workspace_bytes(M, N, K))
    assert 0 < worst <= cap
