"""Operand tiles loaded straight into LDS (LSTMSS_OPT_GEMM_DMA) give the same
bits as the register-staged loads, in both gradient products, through the C
ABI.

Weight gradient: B a multiple of 32 (fp32) or 64 (bf16).  Data gradient:
fp32, K' a multiple of 32.  Rows and columns past the ends of the operands
are clamped to valid ones, so the cases include ragged row groups (H not a
multiple of 16), tiles that end inside the operands (I + H not a multiple of
the tile), several batch chunks per step, several steps per launch and gathered
rows spanning more than one table refill (K' > 2048).  Agreement with the oracle at the default
setting is covered by the parity tests; here both settings must agree bit for
bit on dX, dW, db, dh0, dc0 and the kept indices.  The bf16 weight gradient on
256 x 256 tiles (LSTMSS_OPT_WGRAD_BIG) exists only with DMA chunks and sums in
its own order, so these comparisons switch it off.
"""
import pytest
import torch

from paper_1806_00512_amd.inputs import make_layer

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def L():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_1806_00512_amd.lstmss as lstmss
    lstmss.load()
    return lstmss


def gpu(a, dtype="f32"):
    t = torch.from_numpy(a).to("cuda:0")
    return t.to(torch.bfloat16) if dtype == "bf16" else t


def run_both(L, fn):
    outs = []
    try:
        L.set_option("wgrad_big", 0)
        for dma in (1, 0):
            L.set_option("gemm_dma", dma)
            outs.append(fn())
            torch.cuda.synchronize()
    finally:
        L.set_option("gemm_dma", 1)
        L.set_option("wgrad_big", 1)
    return outs


@pytest.mark.parametrize("T,B,I,H,sp,dtype,struct", [
    (5, 64, 40, 72, 0.5, "f32", {"P": 4, "R": 8}),      # ragged groups, NC = 112
    (4, 128, 96, 64, 0.5, "f32", {"P": 4, "R": 8}),     # 4 chunks per step
    (3, 96, 64, 64, 0.25, "f32", {"P": 2, "R": 8}),     # 3 chunks, two row tiles per group
    (4, 128, 64, 64, 0.0, "f32", None),                 # dense
    (3, 128, 72, 64, 0.5, "bf16", {"P": 4, "R": 8}),    # 2 bf16 chunks per step
    (3, 64, 64, 40, 0.0, "bf16", None),                 # dense bf16, ragged rows
    (3, 128, 64, 64, 0.5, "f32", {"kind": 1, "My": 32, "Mx": 32}),  # 32 x 32 fine blocks
    (3, 70, 40, 64, 0.5, "f32", {"P": 4, "R": 8}),      # ragged B: staged loads either way
    (2, 64, 96, 1096, 0.0, "f32", None),                # dense, K' = 4384 > 2048 gathered rows
    (2, 32, 64, 1088, 0.25, "f32", {"P": 4, "R": 8}),   # K' = 3264: table refills, ragged tiles
    (3, 20, 40, 72, 0.5, "f32", {"P": 4, "R": 8}),      # K' = 144: a 16-row tail, staged either way
    (2, 128, 64, 1088, 0.5, "bf16", {"P": 4, "R": 8}),  # bf16, K' = 2176: splits and a table refill
])
def test_gemm_dma_same_bits(L, T, B, I, H, sp, dtype, struct):
    d = make_layer(T, B, I, H, seed=11 * T + B + H, w_scale=0.2, dtype=dtype, state=True)
    x, W = gpu(d["x"], dtype), gpu(d["W"], dtype)
    dH = gpu(d["dH_up"])
    dhT, dcT = gpu(d["dhT"]), gpu(d["dcT"])
    _, cache = L.fwd_cache(x, W, gpu(d["b"]), gpu(d["h0"]), gpu(d["c0"]))
    torch.cuda.synchronize()
    if struct is None:
        outs = run_both(L, lambda: L.bwd_dense(x, W, cache, dH, dhT=dhT, dcT=dcT))
        keys = ("dX", "dW", "db", "dh0", "dc0")
    else:
        kw = dict(struct)
        outs = run_both(L, lambda: L.bwd_structsparse(x, W, cache, dH, sparsity=sp, dhT=dhT,
                                                      dcT=dcT, **kw))
        keys = ("dX", "dW", "db", "dh0", "dc0", "idx")
    for k in keys:
        assert torch.equal(outs[0][k], outs[1][k]), k
    assert torch.isfinite(outs[0]["dW"]).all()


def test_gemm_dma_stack_same_bits(L):
    # a two-layer stack call: the weight gradient runs in chunks of steps that
    # continue from the stored dW
    T, B, H, I0 = 14, 64, 64, 48
    ds, xs, Ws, caches = [], [], [], []
    inp = None
    for l in range(2):
        I = I0 if l == 0 else H
        d = make_layer(T, B, I, H, seed=40 + l, w_scale=0.2)
        x = gpu(d["x"]) if l == 0 else inp
        W = gpu(d["W"])
        h_out, cache = L.fwd_cache(x, W, gpu(d["b"]))
        xs.append(x); Ws.append(W); caches.append(cache); ds.append(d)
        inp = h_out
    dH = gpu(ds[-1]["dH_up"])
    torch.cuda.synchronize()

    def call():
        dWs = [torch.empty_like(w, dtype=torch.float32) for w in Ws]
        dbs = [torch.empty(w.shape[0], dtype=torch.float32, device="cuda:0") for w in Ws]
        dXs = [None, torch.empty((T, H, B), dtype=torch.float32, device="cuda:0")]
        L.bwd_stack(xs, Ws, caches, dH, sparsity=0.5, dXs=dXs, dWs=dWs, dbs=dbs)
        return dWs + dbs + dXs[1:]

    a, b = run_both(L, call)
    for u, v in zip(a, b):
        assert torch.equal(u, v)


@pytest.mark.parametrize("T,B,I,H,dtype", [
    (4, 64, 96, 64, "f32"),     # both forward products take DMA stages
    (3, 128, 40, 96, "f32"),    # I not a multiple of 32: staged input projection
    (3, 128, 64, 128, "bf16"),  # 128 x 128 bf16 tiles
    (2, 128, 72, 64, "bf16"),   # I not a multiple of 64: staged input projection
])
def test_gemm_dma_forward_same_bits(L, T, B, I, H, dtype):
    d = make_layer(T, B, I, H, seed=3 * T + B + I, w_scale=0.2, dtype=dtype, state=True)
    x, W = gpu(d["x"], dtype), gpu(d["W"], dtype)
    args = (x, W, gpu(d["b"]), gpu(d["h0"]), gpu(d["c0"]))
    outs = run_both(L, lambda: L.fwd_cache(*args))
    assert torch.equal(outs[0][0], outs[1][0])
    assert torch.equal(outs[0][1], outs[1][1])
    assert torch.isfinite(outs[0][0].float()).all()


def test_gemm_dma_misaligned_operands_fall_back(L):
    # an input that starts 4 bytes into its allocation cannot be copied in
    # 16-byte pieces: the products stage it through registers, same bits
    T, B, I, H = 3, 64, 96, 64
    d = make_layer(T, B, I, H, seed=77, w_scale=0.2, state=True)
    x = gpu(d["x"])
    buf = torch.empty(x.numel() + 1, dtype=x.dtype, device=x.device)
    xm = buf[1:].view(T, I, B)
    xm.copy_(x)
    assert xm.data_ptr() % 16 != 0
    W, dH = gpu(d["W"]), gpu(d["dH_up"])
    _, cache = L.fwd_cache(x, W, gpu(d["b"]), gpu(d["h0"]), gpu(d["c0"]))
    _, cache_m = L.fwd_cache(xm, W, gpu(d["b"]), gpu(d["h0"]), gpu(d["c0"]))
    torch.cuda.synchronize()
    assert torch.equal(cache, cache_m)
    a = L.bwd_structsparse(x, W, cache, dH, sparsity=0.5)
    b = L.bwd_structsparse(xm, W, cache_m, dH, sparsity=0.5)
    torch.cuda.synchronize()
    for k in ("dX", "dW", "db", "dh0", "dc0", "idx"):
        assert torch.equal(a[k], b[k]), k
