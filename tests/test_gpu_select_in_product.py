"""GPU: the coarse selection done inside the per-step dh product (option
gemm_select = 1, the default) against the selection kernel launched on its
own (gemm_select = 0).  Every output of a backward call must carry the same
bits at shapes of the two-kernel gate path (H * B >= 65536): splits of whole
regions over 25, 50 and 75 % sparsity, a trailing partial region in the last
split, small and large regions, the chunk sums read directly or staged
through LDS (16 or more per slice), fp32 and bf16; one shape is also checked
against the oracle with the call's own masks."""
import numpy as np
import pytest
import torch

import oracle
from paper_1806_00512_amd.inputs import make_layer

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def L():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_1806_00512_amd.lstmss as lstmss
    lstmss.load()
    return lstmss


def run(L, d, dtype, sparsity, P, R, select_in_product, graphs=True):
    dev = torch.device("cuda:0")

    def g(a):
        t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(dev)
        return t.to(torch.bfloat16) if dtype == "bf16" else t
    x, W = g(d["x"]), g(d["W"])
    dH = torch.from_numpy(np.ascontiguousarray(d["dH_up"], np.float32)).to(dev)
    L.set_option("gemm_select", 1 if select_in_product else 0)
    L.graphs_enable(graphs)
    try:
        _, cache = L.fwd_cache(x, W)
        o = L.bwd_structsparse(x, W, cache, dH, sparsity=sparsity, P=P, R=R, want_dbg=True)
        torch.cuda.synchronize()
    finally:
        L.set_option("gemm_select", 1)
        L.graphs_enable(True)
    return o


SHAPES = [
    # T, B, I, H, sparsity, P, R, dtype
    (3, 128, 256, 512, 0.5, 4, 8, "f32"),     # 8 splits of 128 kept rows
    (3, 64, 1041, 1039, 0.5, 4, 8, "f32"),    # 1039 slices: the last region has 7, 11 splits
    (2, 128, 512, 1024, 0.25, 4, 8, "f32"),   # 16 splits of 192 kept rows (8 regions)
    (2, 256, 128, 256, 0.75, 4, 4, "f32"),    # one kept slice per region, 4 column chunks
    (2, 192, 128, 512, 0.5, 4, 8, "f32"),     # 3 column chunks
    (2, 128, 256, 512, 0.5, 4, 16, "f32"),    # 16-slice regions
    (2, 128, 256, 512, 0.5, 2, 4, "f32"),     # R * P = 8
    (2, 128, 256, 512, 0.5, 1, 8, "f32"),     # one-row slices
    (2, 128, 256, 512, 0.5, 8, 8, "f32"),     # 8-row slices
    (2, 192, 128, 512, 0.5, 8, 8, "f32"),     # 24 chunk sums per slice staged through LDS
    (2, 256, 128, 256, 0.5, 16, 4, "f32"),    # 64 per slice: no room in LDS, direct reads
    (3, 128, 256, 512, 0.5, 4, 8, "bf16"),    # 128 x 128 bf16 tiles, eight wavefronts
    (2, 256, 512, 1024, 0.25, 4, 8, "bf16"),
]


@pytest.mark.parametrize("T,B,I,H,sp,P,R,dtype", SHAPES)
def test_same_bits_as_selection_kernel(L, T, B, I, H, sp, P, R, dtype):
    info = L.bwd_info(L.dims(T, B, I, H, dtype), sp, L.structure(P, R))
    assert info == {"split_gates": True, "select_in_product": True}
    d = make_layer(T, B, I, H, seed=H + B + T, w_scale=0.1, dtype=dtype)
    a = run(L, d, dtype, sp, P, R, True)
    b = run(L, d, dtype, sp, P, R, False)
    for k in ("dX", "dW", "db", "idx", "dbg"):
        assert torch.equal(a[k], b[k]), k


def test_same_bits_without_graphs(L):
    T, B, I, H = 2, 128, 256, 512
    d = make_layer(T, B, I, H, seed=5, w_scale=0.1)
    a = run(L, d, "f32", 0.5, 4, 8, True, graphs=False)
    b = run(L, d, "f32", 0.5, 4, 8, False, graphs=False)
    for k in ("dX", "dW", "db", "idx"):
        assert torch.equal(a[k], b[k]), k


def test_partial_region_against_oracle(L):
    """1039 slices (last region of 7 keeps 4): the masks re-selected by the
    oracle from the call's own pre-sparsify gate gradients, and the gradients
    against the oracle run with those masks (rel. L2 <= 1e-5)."""
    T, B, I, H, P, R, S = 2, 64, 1041, 1039, 4, 8, 4
    d = make_layer(T, B, I, H, seed=7, w_scale=0.1)
    o = run(L, d, "f32", 0.5, P, R, True)
    idx = o["idx"].cpu().numpy()
    dbg = o["dbg"].double().cpu().numpy()
    keep = np.zeros((T, 4 * H // P), np.uint8)
    for t in range(T):
        k = oracle.select(oracle.scores(dbg[t], P), R, S)
        assert np.array_equal(oracle.kept_index(k), idx[t]), t
        keep[t] = k
    x = d["x"].astype(np.float64)
    W = d["W"].astype(np.float64)
    gates, c, h = oracle.forward(x, W)
    ref = oracle.backward(x, W, gates, c, h, d["dH_up"].astype(np.float64), P=P, R=R, S=S,
                          forced_keep=keep)
    for k in ("dW", "db", "dX"):
        a = o[k].double().cpu().numpy()
        e = np.linalg.norm(a - ref[k]) / max(np.linalg.norm(ref[k]), 1e-300)
        assert e <= 1e-5, (k, e)
