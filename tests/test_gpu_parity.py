"""GPU parity: the HIP path (through the C ABI) against the CPU oracle.

Protocol for masks and gradients:
  1. standalone selection: the same gate-gradient bytes go to the GPU
     selector and to the oracle selector -> scores, kept indices and the
     compacted rows must be bit-exact;
  2. in situ: the GPU's own pre-sparsify gate gradient of every step (the
     debug dump) re-selected by the oracle must give the GPU's indices exactly;
  3. gradients: the oracle run with the GPU's masks must match dX, dW, db,
     dh0, dc0 to rel. L2 <= 1e-5 (fp32) / 2e-2 (bf16);
  4. the oracle with its own masks may only disagree on near-ties.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_1806_00512_amd.inputs import WORKLOADS, make_inputs, make_layer

pytestmark = pytest.mark.gpu

TOL = {"f32": 1e-5, "bf16": 2e-2}
NEAR_TIE = {"f32": 1e-5, "bf16": 5e-2}


@pytest.fixture(scope="module")
def L():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_1806_00512_amd.lstmss as lstmss
    lstmss.load()
    return lstmss


def dev():
    return torch.device("cuda:0")


def rel(a, b):
    a, b = np.asarray(a, np.float64), np.asarray(b, np.float64)
    n = np.linalg.norm(b)
    return float(np.linalg.norm(a - b) / (n if n > 0 else 1.0))


def to_np64(t):
    return t.detach().float().cpu().numpy().astype(np.float64)


def gpu_tensor(a, dtype="f32"):
    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(dev())
    return t.to(torch.bfloat16) if dtype == "bf16" else t


def keep_from_idx(idx, nslices):
    keep = np.zeros((idx.shape[0], nslices), np.uint8)
    for t in range(idx.shape[0]):
        keep[t, idx[t]] = 1
    return keep


def check_layer(L, d, dtype, sparsity, P=4, R=8, state=False, dense=False, own=True):
    """Run GPU forward + backward of one layer; check it against the oracle.
    own=False skips the second oracle run with the oracle's own masks (the
    near-tie report), for shapes where one oracle pass takes tens of seconds."""
    T, I, B = d["x"].shape
    H = d["W"].shape[0] // 4
    bf16 = dtype == "bf16"
    x, W = gpu_tensor(d["x"], dtype), gpu_tensor(d["W"], dtype)
    b = gpu_tensor(d["b"]) if d.get("b") is not None else None
    h0 = gpu_tensor(d["h0"]) if d.get("h0") is not None else None
    c0 = gpu_tensor(d["c0"]) if d.get("c0") is not None else None
    dH = gpu_tensor(d["dH_up"])
    dhT = gpu_tensor(d["dhT"]) if d.get("dhT") is not None else None
    dcT = gpu_tensor(d["dcT"]) if d.get("dcT") is not None else None
    h_out, cache = L.fwd_cache(x, W, b, h0, c0)
    if dense:
        o = L.bwd_dense(x, W, cache, dH, dhT, dcT)
    else:
        o = L.bwd_structsparse(x, W, cache, dH, sparsity=sparsity, P=P, R=R, dhT=dhT, dcT=dcT,
                               want_dbg=True)
    torch.cuda.synchronize()

    # forward
    gates, c, h = oracle.forward(d["x"], d["W"], d.get("b"), d.get("h0"), d.get("c0"), bf16=bf16)
    g_gpu, c_gpu, h_gpu = L.cache_views(cache, T, B, H, dtype)
    ftol = 1e-5 if not bf16 else 2e-2
    assert rel(to_np64(h_out), h[1:]) <= ftol
    assert rel(to_np64(c_gpu), c) <= ftol
    assert rel(to_np64(g_gpu), gates) <= ftol

    S = 0 if dense else int(round(sparsity * R))
    nsl = 4 * H // P
    if dense:
        keep = None
    else:
        idx = o["idx"].cpu().numpy()
        dbg = to_np64(o["dbg"])
        # in-situ mask check on the GPU's own gate gradient (bit-exact)
        for t in range(T):
            k = oracle.select(oracle.scores(dbg[t], P), R, S)
            assert np.array_equal(oracle.kept_index(k), idx[t]), "step %d" % t
        keep = keep_from_idx(idx, nsl)
        assert np.all(keep.sum(1) * P == oracle.kept_rows(4 * H, P, R, S))
    ref = oracle.backward(d["x"], d["W"], gates, c, h, d["dH_up"], d.get("dhT"), d.get("dcT"),
                          P=P if not dense else 4, R=R if not dense else 8, S=S, bf16=bf16,
                          forced_keep=keep)
    for k in ("dX", "dW", "db", "dh0", "dc0"):
        e = rel(to_np64(o[k]), ref[k])
        assert e <= TOL[dtype], "%s rel L2 %.3g" % (k, e)
    if not dense and own:
        mine = oracle.backward(d["x"], d["W"], gates, c, h, d["dH_up"], d.get("dhT"), d.get("dcT"),
                               P=P, R=R, S=S, bf16=bf16, want_dG=True)
        mism = np.argwhere(mine["keep"] != keep)
        for t, j in mism:
            sc = oracle.scores(mine["dG"][t], P)
            r0 = (j // R) * R
            reg = sc[r0:r0 + R]
            kept = reg[mine["keep"][t, r0:r0 + R] == 1]
            gap = (kept.min() - np.sort(reg)[::-1][len(kept)]) / max(kept.min(), 1e-300)
            assert gap <= NEAR_TIE[dtype], (t, j, gap)
    return o


# ---------------------------------------------------------------------------
# standalone selection: identical bytes in, bit-exact out
# ---------------------------------------------------------------------------
def adversarial_dG(H, B, P, seed, dtype):
    rng = np.random.default_rng(seed)
    G = 4 * H
    dG = (rng.standard_normal((G, B)) * np.exp(rng.uniform(-3, 3, (G, 1)))).astype(np.float32)
    nsl = G // P
    if nsl >= 8:
        dG[0:P] = 0.0                                  # an all-zero slice
        dG[2 * P:3 * P] = 0.0                          # two tied zero slices
        dG[4 * P:5 * P] = dG[5 * P:6 * P]              # duplicated slice
        perm = rng.permutation(B)
        dG[6 * P:7 * P] = dG[7 * P:8 * P][:, perm]     # same values, permuted columns
    if dtype == "bf16":
        dG = torch.from_numpy(dG).to(torch.bfloat16).float().numpy()
    return dG


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("H,B,P,R,sp", [
    (128, 16, 4, 8, 0.5), (650, 20, 4, 8, 0.5), (72, 70, 4, 8, 0.25), (64, 64, 4, 8, 0.75),
    (256, 256, 4, 8, 0.5), (50, 1, 4, 4, 0.5), (96, 130, 2, 16, 0.5), (33, 33, 1, 5, 0.4),
    (128, 64, 4, 32, 0.5), (64, 48, 4, 64, 0.5)])
def test_select_compact_bit_exact(L, dtype, H, B, P, R, sp):
    dG = adversarial_dG(H, B, P, H * 7 + B, dtype)
    dGc, idx, sc = L.select_compact(gpu_tensor(dG, dtype), sparsity=sp, P=P, R=R)
    torch.cuda.synchronize()
    S = int(round(sp * R))
    ref_sc = oracle.scores(dG.astype(np.float64), P)
    assert np.array_equal(sc.cpu().numpy(), ref_sc)
    keep = oracle.select(ref_sc, R, S)
    ref_idx = oracle.kept_index(keep)
    assert np.array_equal(idx.cpu().numpy(), ref_idx)
    rows = (ref_idx[:, None] * P + np.arange(P)).ravel()
    assert np.array_equal(dGc.float().cpu().numpy(), dG[rows])


def adversarial_regions(H, B, P, R, seed, dtype):
    """Exact ties in every region group and every work-group: whole regions of
    zeros, zero and duplicated slices, regions of identical slices, slices
    that are column permutations of one another (their fp64 sums differ only
    through the fixed summation order), and one NaN slice; the rows' scales
    vary over six orders of magnitude."""
    rng = np.random.default_rng(seed)
    G = 4 * H
    nsl = G // P
    dG = (rng.standard_normal((G, B)) * np.exp(rng.uniform(-3, 3, (G, 1)))).astype(np.float32)

    def sl(j):
        return slice(j * P, (j + 1) * P)
    for r0 in range(0, nsl, R):
        n = min(R, nsl - r0)
        kind = (r0 // R) % 5
        if kind == 0 and n >= 2:
            dG[r0 * P:(r0 + n) * P] = 0.0
        elif kind == 1 and n >= 3:
            dG[sl(r0)] = 0.0
            dG[sl(r0 + 2)] = 0.0
            dG[sl(r0 + 1)] = dG[sl(r0 + n - 1)]
        elif kind == 2 and n >= 2:
            for j in range(1, n):
                dG[sl(r0 + j)] = dG[sl(r0)]
        elif kind == 3 and n >= 2:
            for j in range(1, n):
                dG[sl(r0 + j)] = dG[sl(r0)][:, rng.permutation(B)]
    dG[(nsl // 2) * P + P // 2, B // 3] = np.nan
    if dtype == "bf16":
        dG = torch.from_numpy(dG).to(torch.bfloat16).float().numpy()
    return dG


@pytest.mark.parametrize("H,B,P,R,sp,dtype", [
    (2048, 128, 4, 8, 0.5, "f32"),     # the 4-layer workload's layer shape
    (4096, 256, 4, 8, 0.5, "bf16"),    # the bf16 H = 4096 workload's shape
    (260, 256, 4, 8, 0.5, "f32"),      # regions straddle gate blocks, partial last region
    (256, 256, 4, 8, 0.25, "bf16"),
    (1024, 64, 4, 8, 0.75, "f32"),     # H*B = 65536 exactly
    (512, 128, 4, 4, 0.5, "f32"),      # two regions per select work-group
    (2048, 128, 2, 16, 0.5, "f32"),
    (520, 128, 1, 64, 0.5, "f32"),     # 64-slice regions, partial last region of 32
    (2056, 128, 4, 8, 0.5, "f32"),     # H not a multiple of P*R
    (4104, 256, 4, 8, 0.5, "bf16"),
    (1024, 256, 16, 4, 0.25, "f32"),   # four 64-column chunks, 64-row slices
])
def test_select_split_path_bit_exact(L, H, B, P, R, sp, dtype):
    """Standalone selection on the two-kernel path the backward pass takes at
    H*B >= 65536 (element kernel + select kernel), on adversarial ties: scores,
    kept indices and the compacted rows bit for bit."""
    d = L.dims(1, B, 1, H, dtype)
    assert L.select_workspace_bytes(d, sp, L.structure(P, R)) > 0   # the split path
    dGt = gpu_tensor(adversarial_regions(H, B, P, R, H + B + R, dtype), dtype)
    dG = dGt.float().cpu().numpy()   # the exact bytes the GPU selects on (NaN payload too)
    dGc, idx, sc = L.select_compact(dGt, sparsity=sp, P=P, R=R)
    torch.cuda.synchronize()
    S = int(round(sp * R))
    ref_sc = oracle.scores(dG.astype(np.float64), P)
    got_sc = sc.cpu().numpy()
    assert np.array_equal(got_sc.view(np.uint64)[~np.isnan(ref_sc)],
                          ref_sc.view(np.uint64)[~np.isnan(ref_sc)])
    assert np.array_equal(np.isnan(got_sc), np.isnan(ref_sc))
    ref_idx = oracle.kept_index(oracle.select(ref_sc, R, S))
    assert np.array_equal(idx.cpu().numpy(), ref_idx)
    rows = (ref_idx[:, None] * P + np.arange(P)).ravel()
    got = dGc.float().cpu().numpy()
    assert np.array_equal(got.view(np.uint32), dG[rows].view(np.uint32))


@pytest.mark.parametrize("T,B,I,H,dtype", [
    (2, 256, 32, 256, "f32"), (2, 256, 24, 260, "f32"), (2, 256, 64, 256, "bf16"),
    (2, 128, 40, 1000, "f32")])
def test_split_path_exact_ties_in_situ(L, T, B, I, H, dtype):
    """W = 0, no bias, zero initial state: the i, f and o rows of every gate
    gradient are exactly zero, so every region inside those gate blocks is
    a tie of R zero slices (keep the first R - S), at shapes that run the
    two-kernel gate path; masks in situ bit-exact, gradients to tolerance."""
    d = make_layer(T, B, I, H, seed=H + B, w_scale=0.0, dtype=dtype)
    d["W"] = np.zeros_like(d["W"])
    d["b"] = None
    P, R, S = 4, 8, 4
    o = check_layer(L, d, dtype, 0.5, P=P, R=R)
    idx = o["idx"].cpu().numpy()
    nsl = 4 * H // P

    def zero_slice(j):   # every row of the slice in the i, f or o block
        return all(r < 2 * H or r >= 3 * H for r in range(j * P, j * P + P))
    tied = 0
    for k, r0 in enumerate(range(0, nsl, R)):
        n = min(R, nsl - r0)
        if not all(zero_slice(j) for j in range(r0, r0 + n)):
            continue
        keep = n - S * n // R
        for t in range(T):
            assert np.array_equal(idx[t][k * (R - S):k * (R - S) + keep],
                                  np.arange(r0, r0 + keep)), (t, r0)
        tied += 1
    assert tied >= nsl // R // 2


def test_select_nan_is_kept(L):
    H, B, P, R = 16, 8, 4, 8
    dG = adversarial_dG(H, B, P, 3, "f32")
    dG[3 * P + 1, 5] = np.nan
    _, idx, sc = L.select_compact(gpu_tensor(dG), sparsity=0.75, P=P, R=R)
    torch.cuda.synchronize()
    ref = oracle.kept_index(oracle.select(oracle.scores(dG.astype(np.float64), P), R, 6))
    assert np.array_equal(idx.cpu().numpy(), ref) and 3 in ref


# ---------------------------------------------------------------------------
# end-to-end layer parity
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("T,B,I,H,sp,R,state", [
    (5, 20, 100, 72, 0.5, 8, False),    # ragged everywhere, regions straddle gate blocks
    (4, 70, 64, 64, 0.25, 8, True),     # B above one 64-lane pass, initial state and dhT/dcT
    (3, 16, 33, 40, 0.75, 4, False),
    (2, 1, 8, 8, 0.5, 8, True),         # batch of one
    (1, 32, 128, 128, 0.5, 8, False),   # one step
    (3, 20, 24, 64, 0.25, 16, False),   # 48 kept rows per region: two routing tiles
    (2, 8, 16, 64, 0.5, 64, False),     # 128 kept rows per region: per-step weight gradient
    (2, 256, 32, 64, 0.5, 8, True),     # four 64-column passes per row
    (3, 200, 40, 32, 0.75, 8, False),   # ragged last pass
    (2, 130, 16, 96, 0.5, 2, False),    # small regions (R*P = 8)
])
def test_layer_sparse_f32(L, T, B, I, H, sp, R, state):
    d = make_layer(T, B, I, H, seed=T * 100 + H, w_scale=0.2, state=state)
    check_layer(L, d, "f32", sp, R=R)


@pytest.mark.parametrize("T,B,I,H,sp,R,dtype,dense", [
    (2, 256, 32, 256, 0.5, 8, "f32", False),     # H*B = 65536: split gate kernels
    (3, 200, 40, 400, 0.25, 8, "f32", False),    # ragged last batch chunk
    (2, 256, 24, 260, 0.5, 8, "f32", False),     # unaligned H: regions straddle gates, partial region
    (2, 256, 64, 256, 0.5, 8, "bf16", False),
    (2, 128, 48, 512, 0.75, 4, "f32", False),
    (2, 256, 64, 256, 0.25, 8, "bf16", False),   # 24 kept rows per region: weight-gradient groups
                                                  # of four regions fill three 32-row tiles
    (2, 128, 48, 512, 0.25, 4, "f32", False),    # R = 4, S = 1: 12 kept rows, eight-region groups
    (2, 256, 24, 260, 0.25, 8, "f32", False),    # the last four-region group partial
    (2, 256, 32, 256, 0.0, 8, "f32", True),
    (2, 256, 32, 256, 0.0, 8, "bf16", True),
])
def test_layer_split_path(L, T, B, I, H, sp, R, dtype, dense):
    d = make_layer(T, B, I, H, seed=T + B + H, w_scale=0.1, dtype=dtype, state=True)
    check_layer(L, d, dtype, sp, R=R, dense=dense)


@pytest.mark.parametrize("T,B,I,H", [(5, 20, 100, 72), (3, 150, 40, 64)])
def test_layer_dense_f32(L, T, B, I, H):
    d = make_layer(T, B, I, H, seed=9 + B, w_scale=0.2, state=True)
    check_layer(L, d, "f32", 0.0, dense=True)


@pytest.mark.parametrize("T,B,I,H", [(4, 40, 64, 96), (3, 20, 36, 72)])
def test_layer_sparse_bf16(L, T, B, I, H):
    d = make_layer(T, B, I, H, seed=10 + B, w_scale=0.2, dtype="bf16")
    check_layer(L, d, "bf16", 0.5)


def test_layer_dense_bf16(L):
    d = make_layer(3, 24, 40, 64, seed=13, w_scale=0.2, dtype="bf16", state=True)
    check_layer(L, d, "bf16", 0.0, dense=True)


@pytest.mark.parametrize("B,H,dtype", [(256, 256, "f32"), (128, 512, "bf16"), (200, 400, "f32")])
def test_sparsity_zero_equals_dense_large(L, B, H, dtype):
    """At shapes with H*B >= 65536 (two-kernel gate path) the sparse pass with
    nothing removed gives the dense pass's bits."""
    d = make_layer(3, B, 48, H, seed=B + H, w_scale=0.1, dtype=dtype, state=True)
    x, W = gpu_tensor(d["x"], dtype), gpu_tensor(d["W"], dtype)
    dH = gpu_tensor(d["dH_up"])
    dhT, dcT = gpu_tensor(d["dhT"]), gpu_tensor(d["dcT"])
    _, cache = L.fwd_cache(x, W, gpu_tensor(d["b"]), gpu_tensor(d["h0"]), gpu_tensor(d["c0"]))
    a = L.bwd_dense(x, W, cache, dH, dhT, dcT)
    b = L.bwd_structsparse(x, W, cache, dH, sparsity=0.0, P=4, R=8, dhT=dhT, dcT=dcT)
    torch.cuda.synchronize()
    for k in ("dX", "dW", "db", "dh0", "dc0"):
        assert torch.equal(a[k], b[k]), k


def test_sparsity_zero_equals_dense(L):
    d = make_layer(4, 24, 48, 64, seed=11, w_scale=0.2, state=True)
    x, W = gpu_tensor(d["x"]), gpu_tensor(d["W"])
    dH = gpu_tensor(d["dH_up"])
    dhT, dcT = gpu_tensor(d["dhT"]), gpu_tensor(d["dcT"])
    _, cache = L.fwd_cache(x, W, None, gpu_tensor(d["h0"]), gpu_tensor(d["c0"]))
    a = L.bwd_dense(x, W, cache, dH, dhT, dcT)
    b = L.bwd_structsparse(x, W, cache, dH, sparsity=0.0, P=4, R=8, dhT=dhT, dcT=dcT)
    torch.cuda.synchronize()
    for k in ("dX", "dW", "db", "dh0", "dc0"):
        assert torch.equal(a[k], b[k]), k
    assert torch.equal(b["idx"].cpu(), torch.arange(64, dtype=torch.int32).repeat(4, 1))


@pytest.mark.parametrize("H,sp", [(72, 0.5), (64, 0.5), (64, 0.0)])
def test_graph_replay_matches_direct(L, H, sp):
    """Captured-and-replayed calls give the same bits as direct launches,
    on every replay, with other work in between."""
    d = make_layer(4, 20, 40, H, seed=14, w_scale=0.2, state=True)
    x, W, dH = gpu_tensor(d["x"]), gpu_tensor(d["W"]), gpu_tensor(d["dH_up"])
    dhT, dcT = gpu_tensor(d["dhT"]), gpu_tensor(d["dcT"])
    _, cache = L.fwd_cache(x, W)
    L.graphs_enable(False)
    try:
        ref = L.bwd_structsparse(x, W, cache, dH, sp, dhT=dhT, dcT=dcT)
        torch.cuda.synchronize()
    finally:
        L.graphs_enable(True)
    d0 = L.dims(4, 20, 40, H)
    ws = torch.empty(L.workspace_bytes(d0, sp, L.structure(4, 8) if sp else None),
                     dtype=torch.uint8, device=dev())
    out = {k: torch.empty_like(v) for k, v in ref.items() if v is not None}
    for rep in range(3):
        for v in out.values():
            v.fill_(float("nan") if v.dtype.is_floating_point else -7)
        torch.cuda.synchronize()
        o = L.bwd_structsparse(x, W, cache, dH, sp, dhT=dhT, dcT=dcT, out=out, ws=ws)
        torch.cuda.synchronize()
        for k in ("dX", "dW", "db", "dh0", "dc0", "idx"):
            assert torch.equal(o[k], ref[k]), (rep, k)
        torch.randn(1000, device=dev()).sum().item()  # unrelated eager work between replays


@pytest.mark.parametrize("T,B,I,H,sp,big", [
    (3, 64, 1024, 2048, 0.5, 1),     # 256 x 256 tiles, 128 kept rows each
    (3, 64, 1024, 2048, 0.5, 0),     # the routing kernel on the same shape
    (3, 64, 1000, 2050, 0.25, 1),    # 192 kept rows; ragged tiles, a partial last region
    (3, 128, 1000, 2050, 0.0, 1),    # dense, ragged tiles
    (3, 64, 1024, 2048, 0.75, 1),    # 64 kept rows per tile: the routing kernel
    (3, 64, 512, 512, 0.5, 1),       # 32 tiles, fewer than 256: the routing kernel
])
def test_wgrad_big_bf16(L, T, B, I, H, sp, big):
    """The bf16 weight gradient on 256-row x 256-feature tiles (dropped rows
    multiplied as zeros) and the kernel that routes the kept rows' products,
    each against the oracle."""
    d = make_layer(T, B, I, H, seed=T + B + H, w_scale=0.1, dtype="bf16", state=True)
    try:
        L.set_option("wgrad_big", big)
        check_layer(L, d, "bf16", sp, dense=sp == 0.0, own=False)
    finally:
        L.set_option("wgrad_big", 1)


def test_side_stream_modes_identical_bf16_big(L):
    """Steps of the 256 x 256-tile bf16 weight gradient split over side-stream
    launches (each continuing the stored sums) give the bits of one launch."""
    d = make_layer(20, 64, 1024, 2048, seed=16, w_scale=0.1, dtype="bf16", state=True)
    x, W = gpu_tensor(d["x"], "bf16"), gpu_tensor(d["W"], "bf16")
    dH, dhT, dcT = gpu_tensor(d["dH_up"]), gpu_tensor(d["dhT"]), gpu_tensor(d["dcT"])
    _, cache = L.fwd_cache(x, W)
    outs = []
    try:
        for mode in (1, 0):
            L.set_option("side_stream", mode)
            outs.append(L.bwd_structsparse(x, W, cache, dH, 0.5, dhT=dhT, dcT=dcT))
            torch.cuda.synchronize()
    finally:
        L.set_option("side_stream", 2)
    for k in ("dX", "dW", "db", "dh0", "dc0", "idx"):
        assert torch.equal(outs[1][k], outs[0][k]), k


@pytest.mark.parametrize("graphs", [True, False])
def test_side_stream_modes_identical(L, graphs):
    """The weight gradient and dX on the side stream (1), in order on the
    caller's stream (0) or chosen by shape (2) give the same bits."""
    d = make_layer(20, 64, 96, 128, seed=15, w_scale=0.2, state=True)
    x, W, dH = gpu_tensor(d["x"]), gpu_tensor(d["W"]), gpu_tensor(d["dH_up"])
    dhT, dcT = gpu_tensor(d["dhT"]), gpu_tensor(d["dcT"])
    _, cache = L.fwd_cache(x, W)
    outs = []
    try:
        L.graphs_enable(graphs)
        for mode in (1, 0, 2):
            L.set_option("side_stream", mode)
            outs.append(L.bwd_structsparse(x, W, cache, dH, 0.5, dhT=dhT, dcT=dcT))
            torch.cuda.synchronize()
    finally:
        L.set_option("side_stream", 2)
        L.graphs_enable(True)
    for o in outs[1:]:
        for k in ("dX", "dW", "db", "dh0", "dc0", "idx"):
            assert torch.equal(o[k], outs[0][k]), k
    with pytest.raises(L.LstmssError):
        L.set_option("side_stream", 3)


def test_deterministic(L):
    d = make_layer(4, 20, 40, 64, seed=12, w_scale=0.2)
    x, W, dH = gpu_tensor(d["x"]), gpu_tensor(d["W"]), gpu_tensor(d["dH_up"])
    _, cache = L.fwd_cache(x, W)
    a = L.bwd_structsparse(x, W, cache, dH, 0.5)
    b = L.bwd_structsparse(x, W, cache, dH, 0.5)
    torch.cuda.synchronize()
    for k in ("dX", "dW", "db", "dh0", "dc0", "idx"):
        assert torch.equal(a[k], b[k]), k


@pytest.mark.parametrize("name,steps", [
    ("lstm1_h128_b16_t20_f32", None),
    ("lstm2_lm_h650_b20_t35_f32", None),
    ("lstm2_h1024_b64_t35_f32", None),
    ("lstm4_enc_h2048_b128_t50_f32", 4),    # full H and B, all four layers, T cut to 4
])
def test_workload_full(L, name, steps):
    """Workloads at full layer size, every layer (top layer first)."""
    wl = WORKLOADS[name] if steps is None else WORKLOADS[name].truncated(steps)
    inp = make_inputs(wl, seed=0)
    caches = oracle.stack_forward(inp["x"], inp["Ws"])
    up = inp["dH_up"]
    layer_x = [inp["x"]] + [cc["h"][1:] for cc in caches[:-1]]
    for li in reversed(range(wl.layers)):
        # each layer is checked with the oracle's own input and upstream
        # gradient, so that errors do not compound across layers
        d = {"x": layer_x[li].astype(np.float32), "W": inp["Ws"][li], "b": None,
             "dH_up": np.asarray(up, np.float32)}
        o = check_layer(L, d, wl.dtype, wl.sparsity, P=wl.P, R=wl.R, own=wl.hidden <= 1024)
        if li == 0:
            break
        ref = oracle.backward(caches[li]["x"], caches[li]["W"], caches[li]["gates"],
                              caches[li]["c"], caches[li]["h"], up, P=wl.P, R=wl.R,
                              S=int(round(wl.sparsity * wl.R)),
                              forced_keep=keep_from_idx(o["idx"].cpu().numpy(),
                                                        4 * wl.hidden // wl.P))
        up = ref["dX"]


@pytest.mark.parametrize("sp", [0.0, 0.25, 0.75])
def test_sparsity_sweep_h1024(L, sp):
    """The sweep of the 2-layer H = 1024 workload at full size (bottom layer)."""
    wl = WORKLOADS["lstm2_h1024_b64_t35_f32"]
    inp = make_inputs(wl, seed=0)
    d = {"x": inp["x"], "W": inp["Ws"][0], "b": None, "dH_up": inp["dH_up"]}
    check_layer(L, d, wl.dtype, sp, P=wl.P, R=wl.R)


def test_full_length_h2048(L):
    """Bottom layer of the 4-layer H = 2048 workload over all 50 steps as one
    single-layer call (graph replay, the split gate kernels, one weight-
    gradient and input-gradient launch each, in order on the caller's
    stream).  The benchmark's own call, the four-layer stack, is checked
    against the oracle in test_gpu_stack.py."""
    wl = WORKLOADS["lstm4_enc_h2048_b128_t50_f32"]
    inp = make_inputs(wl, seed=0)
    d = {"x": inp["x"], "W": inp["Ws"][0], "b": None, "dH_up": inp["dH_up"]}
    check_layer(L, d, wl.dtype, wl.sparsity, P=wl.P, R=wl.R, own=False)


def test_bf16_h4096(L):
    """The bf16 H = 4096, B = 256 layer at full size with T cut to 4."""
    wl = WORKLOADS["lstm1_h4096_b256_t100_bf16"].truncated(4)
    inp = make_inputs(wl, seed=0)
    d = {"x": inp["x"], "W": inp["Ws"][0], "b": None, "dH_up": inp["dH_up"]}
    check_layer(L, d, wl.dtype, wl.sparsity, P=wl.P, R=wl.R, own=False)


@pytest.mark.parametrize("sp", [0.5, 0.0])
def test_bf16_h4096_full_length_sampled(L, sp):
    """The bf16 H = 4096, B = 256, T = 100 layer call as the benchmark makes it
    (one weight-gradient launch over all 100 steps, batched dX launches), at
    50 % and at sparsity 0 (bit-identical to the dense call of the 9 : 1
    schedule):
    sampled entries of dW, dX and db, each summed in fp64 from the GPU's own
    gate gradients, masks and cached inputs (sections 3 and 4: dW sums
    dG_t [x_t; h_{t-1}]^T over the kept rows, dX_t = W_x^T dG_t over the kept
    rows), and the masks of a few steps against the oracle's selection."""
    wl = WORKLOADS["lstm1_h4096_b256_t100_bf16"]
    inp = make_inputs(wl, seed=0)
    T, B, I, H, P, R = wl.steps, wl.batch, wl.input_size, wl.hidden, wl.P, wl.R
    S = int(round(sp * R))
    x, W = gpu_tensor(inp["x"], "bf16"), gpu_tensor(inp["Ws"][0], "bf16")
    dH = gpu_tensor(inp["dH_up"])
    _, cache = L.fwd_cache(x, W)
    o = L.bwd_structsparse(x, W, cache, dH, sparsity=sp, P=P, R=R, want_dbg=True)
    torch.cuda.synchronize()
    _, _, h = L.cache_views(cache, T, B, H, "bf16")
    idx = o["idx"].cpu().numpy()
    keep = keep_from_idx(idx, 4 * H // P)                          # [T][slices]
    assert np.all(keep.sum(1) * P == oracle.kept_rows(4 * H, P, R, S))
    for t in (0, T // 2, T - 1):                                    # masks, bit-exact
        k = oracle.select(oracle.scores(to_np64(o["dbg"][t]), P), R, S)
        assert np.array_equal(oracle.kept_index(k), idx[t]), t
    rng = np.random.default_rng(7)
    n = 48
    rows = torch.from_numpy(rng.integers(0, 4 * H, n)).to(dev())
    cols = rng.integers(0, I + H, n)
    g = o["dbg"].index_select(1, rows).double().cpu().numpy()      # [T][n][B]
    rows = rows.cpu().numpy()
    xh = np.empty((T, n, B))
    for j, c in enumerate(cols):
        src = x[:, c, :] if c < I else h[:T, c - I, :]              # h[t] = h_{t-1}
        xh[:, j, :] = src.double().cpu().numpy()
    kr = keep[:, rows // P].astype(np.float64)                      # [T][n]
    terms = kr[:, :, None] * g * xh
    ref = terms.sum(axis=(0, 2))
    got = o["dW"][torch.from_numpy(rows).to(dev()), torch.from_numpy(cols).to(dev())]
    err = np.abs(got.double().cpu().numpy() - ref)
    mag = np.abs(terms).sum(axis=(0, 2))
    # bf16 x bf16 products are exact in fp32; the fp32 sums of 25600 of them
    # stay far below this bound, while one step missing or misplaced (about a
    # hundredth of a sum of random signs) exceeds it
    print("dW sample error / sum |terms|: max %.3g" % (err / mag).max())
    assert np.all(err <= 2e-5 * mag + 1e-30), (err / mag).max()
    # db: each kept step's row sum
    dbr = (kr[:, :, None] * g).sum(axis=(0, 2))
    assert np.allclose(o["db"][torch.from_numpy(rows).to(dev())].double().cpu().numpy(), dbr,
                       rtol=1e-4, atol=1e-4 * np.abs(kr[:, :, None] * g).sum(axis=(0, 2)).max())
    # dX: sampled (t, i, b) over all kept rows of step t
    ts, ii, bb = rng.integers(0, T, n), rng.integers(0, I, n), rng.integers(0, B, n)
    Wx = W[:, torch.from_numpy(ii).to(dev())].double().cpu().numpy()          # [4H][n]
    for j in range(n):
        t = ts[j]
        gt = o["dbg"][t, :, bb[j]].double().cpu().numpy()                       # [4H]
        m = np.repeat(keep[t], P).astype(np.float64)
        tj = m * gt * Wx[:, j]
        assert abs(o["dX"][t, ii[j], bb[j]].item() - tj.sum()) <= 1e-4 * np.abs(tj).sum() + 1e-30, j


def test_error_paths(L):
    d = L.dims(2, 4, 4, 8)
    assert L.kept_rows(d, 0.5, L.structure(4, 8)) == 16
    with pytest.raises(L.LstmssError):
        L.kept_rows(d, 0.3, L.structure(4, 8))      # 0.3 * 8 is not an integer
    with pytest.raises(L.LstmssError):
        L.kept_rows(d, 0.5, L.structure(3, 8))      # P does not divide 4H
    with pytest.raises(L.LstmssError):
        L.kept_rows(d, 0.5, L.structure(4, 65))     # R > 64
    with pytest.raises(L.LstmssError) as e:
        L.kept_rows(d, 0.5, L.structure(kind=L.FINE, My=16, Mx=0))   # Mx missing
    assert e.value.code == -1
    with pytest.raises(L.LstmssError) as e:
        L.kept_rows(L.dims(2, 512, 4, 8), 0.5, L.structure(kind=L.FINE, My=64, Mx=4))
    assert e.value.code == -2                           # batch above 256 columns
    x = torch.zeros((2, 4, 4), device=dev())
    W = torch.zeros((32, 12), device=dev())
    _, cache = L.fwd_cache(x, W)
    small = torch.empty(16, dtype=torch.uint8, device=dev())
    with pytest.raises(L.LstmssError) as e:
        L.bwd_structsparse(x, W, cache, torch.zeros((2, 8, 4), device=dev()), 0.5, ws=small)
    assert e.value.code == -3
