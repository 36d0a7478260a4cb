"""GPU: the entry point that allocates nothing (lstmss_select_compact_noalloc,
scratch in a static device array) gives the bits of lstmss_select_compact
(caller workspace) on two calls in a row, the second with a smaller input,
and a shape whose scratch would exceed the static array is refused before
any pointer is used."""
import ctypes

import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def L():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_1806_00512_amd.lstmss as lstmss
    lstmss.load()
    return lstmss


def gate_gradient(H, B, seed, dtype):
    """Random rows of varying scale with a few exact ties (zero and duplicated
    slices), stored in the workload's storage type."""
    rng = np.random.default_rng(seed)
    dG = (rng.standard_normal((4 * H, B)) * np.exp(rng.uniform(-2, 2, (4 * H, 1))))
    dG = dG.astype(np.float32)
    dG[0:8] = 0.0
    dG[12:16] = dG[16:20]
    t = torch.from_numpy(dG).to("cuda:0")
    return t.to(torch.bfloat16) if dtype == "bf16" else t


@pytest.mark.parametrize("first,second", [
    ((2048, 128, "f32"), (1024, 64, "f32")),      # both on the two-kernel path
    ((4096, 256, "bf16"), (260, 256, "bf16")),    # the largest workload shape, then a ragged one
    ((2048, 128, "f32"), (128, 16, "f32")),       # then a shape without scratch
])
def test_noalloc_matches_workspace_call(L, first, second):
    for k, (H, B, dtype) in enumerate((first, second)):
        dG = gate_gradient(H, B, seed=H + B + k, dtype=dtype)
        ref_c, ref_i, ref_s = L.select_compact(dG, sparsity=0.5, P=4, R=8)
        torch.cuda.synchronize()
        got_c = torch.full_like(ref_c, float("nan"))
        got_i = torch.full_like(ref_i, -7)
        got_s = torch.full_like(ref_s, float("nan"))
        torch.cuda.synchronize()
        L.select_compact_noalloc(dG, got_c, got_i, got_s, sparsity=0.5, P=4, R=8)
        torch.cuda.synchronize()
        assert torch.equal(got_i, ref_i), (k, H, B)
        assert torch.equal(got_c.view(torch.int16 if dtype == "bf16" else torch.int32),
                           ref_c.view(torch.int16 if dtype == "bf16" else torch.int32)), (k, H, B)
        assert torch.equal(got_s, ref_s), (k, H, B)


def test_noalloc_refuses_oversized_scratch(L):
    """4H * ceil(B/64) * 8 bytes above the static array: refused with
    LSTMSS_ERR_UNSUPPORTED; the pointers are NULL, so nothing could run."""
    H, B = 16384, 256          # 65536 rows x 4 chunks x 8 bytes = 2 MiB
    d = L.dims(1, B, 1, H)
    assert L.select_workspace_bytes(d, 0.5, L.structure(4, 8)) > L.NOALLOC_SCRATCH_BYTES
    s = L.structure(4, 8)
    rc = L.load().lstmss_select_compact_noalloc(ctypes.byref(d), 0.5, ctypes.byref(s), None,
                                                None, None, None, None)
    assert rc == -2
    assert b"static buffer" in L.load().lstmss_last_error()
