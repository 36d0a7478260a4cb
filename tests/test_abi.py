"""CPU-side checks of the C ABI: the library loads, exports every symbol the
header declares, and its host-only entry points (size queries, argument
validation) behave.  No GPU compute is launched here."""
import ctypes
import os
import re

import numpy as np
import pytest

import oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "lstmss.h")


@pytest.fixture(scope="module")
def L():
    import paper_1806_00512_amd.lstmss as lstmss
    lstmss.load()
    return lstmss


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\s*\*?\s*(\w+)\s*\(", text, flags=re.M)))


def test_header_symbols_exported(L):
    names = declared_functions()
    assert "lstm_bwd_structsparse" in names and len(names) >= 10
    lib = ctypes.CDLL(L.LIB_PATH)
    for n in names:
        assert hasattr(lib, n), n
    assert set(L.SYMBOLS) == set(names)
    assert L.load().lstmss_version() == 1


def test_strerror(L):
    lib = L.load()
    assert lib.lstmss_strerror(0) == b"success"
    assert lib.lstmss_strerror(-3) == b"workspace too small"
    assert lib.lstmss_strerror(-99) == b"unknown error code"


@pytest.mark.parametrize("H,P,R,sp", [(128, 4, 8, 0.5), (650, 4, 8, 0.5), (1024, 4, 8, 0.25),
                                      (1024, 4, 8, 0.75), (2048, 4, 8, 0.5), (4096, 4, 8, 0.5),
                                      (650, 2, 16, 0.5), (100, 4, 32, 0.5), (33, 1, 5, 0.4),
                                      (512, 4, 4, 0.5), (512, 4, 64, 0.25)])
def test_kept_rows_matches_oracle(L, H, P, R, sp):
    d = L.dims(3, 16, 32, H)
    S = int(round(sp * R))
    assert L.kept_rows(d, sp, L.structure(P, R)) == oracle.kept_rows(4 * H, P, R, S)
    assert L.kept_rows(d, 0.0, L.structure(P, R)) == 4 * H


def test_sizes(L):
    for dt, es in ((L.F32, 4), (L.BF16, 2)):
        d = L.dims(35, 20, 650, 650, dt)
        cb = L.cache_bytes(d)
        assert cb >= 35 * 4 * 650 * 20 * es + 36 * 650 * 20 * (4 + es)
        wd = L.workspace_bytes(d, 0.0, None)
        ws = L.workspace_bytes(d, 0.5, L.structure(4, 8))
        # the compacted gate gradient of every step dominates the workspace
        assert wd > ws >= 35 * 1300 * 20 * es


@pytest.mark.parametrize("H,B,P,R,sp,split", [
    (2048, 128, 4, 8, 0.5, True), (4096, 256, 4, 8, 0.5, True), (260, 256, 4, 8, 0.5, True),
    (1024, 64, 4, 8, 0.75, True), (128, 16, 4, 8, 0.5, False), (1023, 64, 4, 8, 0.5, False),
    (2048, 128, 4, 128, 0.5, None), (2048, 128, 16, 32, 0.5, False)])
def test_select_workspace(L, H, B, P, R, sp, split):
    """The standalone selection needs scratch exactly where the backward pass
    takes the two-kernel gate path (H*B >= 65536 and a region group that fits
    the select kernel): one fp64 sum of squares per row and 64-column chunk."""
    d = L.dims(1, B, 1, H)
    if split is None:
        with pytest.raises(L.LstmssError):
            L.select_workspace_bytes(d, sp, L.structure(P, R))
        return
    n = L.select_workspace_bytes(d, sp, L.structure(P, R))
    if split:
        assert n >= 4 * H * (-(-B // 64)) * 8 and n % 256 == 0
    else:
        assert n == 0
    assert L.select_workspace_bytes(d, 0.5, L.structure(kind=L.FINE, My=8, Mx=4)) == 0


@pytest.mark.parametrize("args,code", [
    ((0, 4, 4, 8), -1), ((2, 4, 4, -1), -1), ((2, 4, 4, 8, 7), -2)])
def test_bad_dims(L, args, code):
    d = L.Dims(*(list(args) + [0] * (5 - len(args))))
    n = L.load().lstmss_cache_bytes(ctypes.byref(d))
    assert n == code
    assert L.load().lstmss_last_error()


@pytest.mark.parametrize("P,R,sp,code", [(3, 8, 0.5, -1), (4, 0, 0.5, -1), (4, 65, 0.5, -1),
                                         (4, 8, 0.3, -1), (4, 8, 1.0, -1), (4, 8, -0.125, -1),
                                         (4, 8, float("nan"), -1)])
def test_bad_structure(L, P, R, sp, code):
    d = L.dims(2, 4, 4, 8)
    n = L.load().lstmss_kept_rows(ctypes.byref(d), sp, ctypes.byref(L.structure(P, R)))
    assert n == code


@pytest.mark.parametrize("B,My,Mx,sp", [(128, 16, 4, 0.5), (100, 32, 4, 0.25), (256, 32, 2, 0.75),
                                         (20, 4, 8, 0.2), (64, 64, 1, 0.0)])
def test_fine_sizes(L, B, My, Mx, sp):
    """Fine structure: products run on the masked [4H][B] matrix; the index
    lists nb - K kept blocks of every Mx-row slice (section 3, Fig. 2(b))."""
    H = 64
    d = L.dims(3, B, 32, H)
    s = L.structure(kind=L.FINE, My=My, Mx=Mx)
    nb = -(-B // My)
    K = round(sp * nb)
    assert L.kept_rows(d, sp, s) == 4 * H
    assert L.index_entries(d, sp, s) == (4 * H // Mx) * (nb - K)
    assert L.workspace_bytes(d, sp, s) >= 3 * 4 * H * B * 4


@pytest.mark.parametrize("B,My,Mx,sp,code", [
    (128, 16, 3, 0.5, -1),    # Mx does not divide 32
    (128, 16, 64, 0.5, -1),   # Mx above 32
    (128, 12, 4, 0.5, -1),    # My not a power of two
    (128, 1, 4, 0.5, -1),     # My below 2
    (128, 128, 4, 0.5, -1),   # My above 64
    (128, 16, 4, 0.3, -1),    # sparsity * nb not an integer
    (128, 16, 4, 1.0, -1),    # every block removed
    (256, 2, 4, 0.5, -1),     # 128 blocks per slice
    (512, 64, 4, 0.5, -2)])   # batch above the fine kernel's 256 columns
def test_bad_fine_structure(L, B, My, Mx, sp, code):
    d = L.dims(2, B, 4, 8)
    s = L.structure(kind=L.FINE, My=My, Mx=Mx)
    assert L.load().lstmss_kept_rows(ctypes.byref(d), sp, ctypes.byref(s)) == code
    assert L.load().lstmss_index_entries(ctypes.byref(d), sp, ctypes.byref(s)) == code


def test_coarse_index_entries(L):
    d = L.dims(2, 20, 650, 650)
    s = L.structure(4, 8)
    assert L.index_entries(d, 0.5, s) == L.kept_rows(d, 0.5, s) // 4


def test_null_pointers_rejected_before_launch(L):
    lib = L.load()
    d = L.dims(2, 4, 4, 8)
    rc = lib.lstm_fwd_cache(ctypes.byref(d), None, None, None, None, None, None, None, None, 0,
                            None)
    assert rc == -1
    s = L.structure(4, 8)
    rc = lib.lstm_bwd_structsparse(ctypes.byref(d), 0.5, ctypes.byref(s), *([None] * 14), 0, None)
    assert rc == -1
    rc = lib.lstm_bwd_dense(ctypes.byref(d), *([None] * 12), 0, None)
    assert rc == -1
    assert b"NULL" in lib.lstmss_last_error()


def test_product_path_fails_loudly_without_library(tmp_path, monkeypatch):
    import paper_1806_00512_amd.lstmss as lstmss
    monkeypatch.setattr(lstmss, "_lib", None)
    monkeypatch.setattr(lstmss, "LIB_PATH", str(tmp_path / "missing.so"))
    with pytest.raises(RuntimeError):
        lstmss.load()


def test_stack_workspace_and_validation(L):
    lib = L.load()
    s = L.structure(4, 8)
    ds = (L.Dims * 2)(L.dims(4, 8, 16, 32), L.dims(4, 8, 32, 32))
    n = lib.lstmss_stack_workspace_bytes(2, ds, 0.5, ctypes.byref(s))
    assert n >= L.workspace_bytes(ds[0], 0.5, s) + L.workspace_bytes(ds[1], 0.5, s)
    nd = lib.lstmss_stack_workspace_bytes(2, ds, 0.0, None)
    assert nd >= L.workspace_bytes(ds[0]) + L.workspace_bytes(ds[1])
    bad_i = (L.Dims * 2)(L.dims(4, 8, 16, 32), L.dims(4, 8, 16, 32))   # I != H below
    assert lib.lstmss_stack_workspace_bytes(2, bad_i, 0.5, ctypes.byref(s)) == -1
    bad_t = (L.Dims * 2)(L.dims(4, 8, 16, 32), L.dims(5, 8, 32, 32))   # T differs
    assert lib.lstmss_stack_workspace_bytes(2, bad_t, 0.5, ctypes.byref(s)) == -1
    assert lib.lstmss_stack_workspace_bytes(0, ds, 0.5, ctypes.byref(s)) == -1
    assert lib.lstmss_stack_workspace_bytes(9, ds, 0.5, ctypes.byref(s)) == -1
    # pointer checks run before any device work
    null = (ctypes.c_void_p * 2)()
    rc = lib.lstm_bwd_stack(2, ds, 0.5, ctypes.byref(s), null, null, null, None, null, null,
                            None, None, None, 0, None)
    assert rc == -1


def test_bidir_host_checks(L):
    lib = L.load()
    assert lib.lstmss_time_reverse(0, 16, None, None, None) == -1
    assert lib.lstmss_time_reverse(4, 6, None, None, None) == -1      # not a multiple of 4
    d = L.dims(4, 8, 16, 32)
    s = L.structure(4, 8)
    n = lib.lstmss_bidir_workspace_bytes(ctypes.byref(d), 0.5, ctypes.byref(s))
    assert n >= 2 * L.workspace_bytes(d, 0.5, s) + 2 * 4 * 32 * 8 * 4 + 2 * 4 * 16 * 8 * 4
    rc = lib.lstm_bwd_bidir(ctypes.byref(d), 0.5, ctypes.byref(s), *([None] * 15), 0, None)
    assert rc == -1


def test_options_match_header_and_validate(L):
    # the binding's option table is the header's enum; the setter validates
    text = open(HEADER).read()
    enum = dict((k, int(v)) for k, v in re.findall(r"LSTMSS_OPT_(\w+)\s*=\s*(\d+)", text))
    assert {k.lower(): v for k, v in enum.items()} == L.OPTIONS
    lib = L.load()
    defaults = {"graphs": 0 if os.environ.get("LSTMSS_GRAPHS") == "0" else 1, "side_stream": 2,
                "stack_dx_steps": 0, "fine_skip": 1, "gemm_dma": 1, "gemm_select": 1,
                "fine_fused": 1, "wgrad_big": 1}
    assert set(defaults) == set(L.OPTIONS)
    try:
        for name in ("fine_skip", "gemm_dma", "gemm_select", "fine_fused", "wgrad_big", "graphs"):
            for v in (0, 1):
                assert lib.lstmss_set_option(L.OPTIONS[name], v) == 0
        for v in (0, 1, 2):
            assert lib.lstmss_set_option(L.OPTIONS["side_stream"], v) == 0
        assert lib.lstmss_set_option(L.OPTIONS["side_stream"], 3) == -1
        assert lib.lstmss_set_option(L.OPTIONS["stack_dx_steps"], -1) == -1
        assert lib.lstmss_set_option(L.OPTIONS["stack_dx_steps"], 6) == 0
        assert lib.lstmss_set_option(max(L.OPTIONS.values()) + 1, 1) == -1
    finally:
        for name, v in defaults.items():
            assert lib.lstmss_set_option(L.OPTIONS[name], v) == 0


@pytest.mark.parametrize("T,B,I,H,sp,P,R,dtype,split,sel", [
    (50, 128, 2048, 2048, 0.5, 4, 8, "f32", True, True),     # 4-layer encoder shape
    (50, 128, 2048, 2048, 0.25, 4, 8, "f32", True, True),
    (35, 64, 1024, 1024, 0.75, 4, 8, "f32", True, True),
    (100, 256, 4096, 4096, 0.5, 4, 8, "bf16", True, True),
    (3, 64, 1041, 1039, 0.5, 4, 8, "f32", True, True),      # trailing partial region
    (3, 128, 256, 512, 0.5, 8, 8, "f32", True, True),       # 8-row slices
    (3, 320, 64, 256, 0.5, 4, 8, "f32", True, True),        # five column chunks
    (3, 200, 40, 400, 0.25, 4, 8, "f32", True, False),      # K' = 1200: no whole DMA stages
    (20, 16, 128, 128, 0.5, 4, 8, "f32", False, False),     # H * B < 65536: one gate kernel
    (35, 64, 1024, 1024, 0.0, 4, 8, "f32", True, False),    # nothing removed
])
def test_bwd_info(L, T, B, I, H, sp, P, R, dtype, split, sel):
    """Which gate path a backward call takes (host logic, no GPU work); the
    selection leaves the product when the option is off or DMA stages are."""
    d = L.dims(T, B, I, H, dtype)
    s = L.structure(P, R)
    assert L.bwd_info(d, sp, s) == {"split_gates": split, "select_in_product": sel}
    try:
        for opt in ("gemm_select", "gemm_dma"):
            L.set_option(opt, 0)
            assert L.bwd_info(d, sp, s) == {"split_gates": split, "select_in_product": False}
            L.set_option(opt, 1)
    finally:
        L.set_option("gemm_select", 1)
        L.set_option("gemm_dma", 1)
    with pytest.raises(L.LstmssError):
        L.bwd_info(d, 0.3, s)
