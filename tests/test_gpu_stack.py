"""GPU: the wavefront backward of a layer stack (lstm_bwd_stack) gives the
same bits as the layers' backward calls made one after the other, top layer
first; with graphs and without, for the coarse, fine and dense cases; and at
the benchmark's own shape it matches the oracle layer by layer."""
import numpy as np
import pytest
import torch

import oracle
from paper_1806_00512_amd.inputs import WORKLOADS, make_inputs

pytestmark = pytest.mark.gpu


def rel(a, b):
    a = a.double().cpu().numpy() if isinstance(a, torch.Tensor) else np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    n = np.linalg.norm(b)
    return float(np.linalg.norm(a - b) / (n if n > 0 else 1.0))


@pytest.fixture(scope="module")
def L():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_1806_00512_amd.lstmss as lstmss
    lstmss.load()
    return lstmss


def make_stack(L, layers, T, B, I, H, seed, dtype=torch.float32):
    rng = np.random.default_rng(seed)
    dev = torch.device("cuda:0")
    x = torch.from_numpy(rng.standard_normal((T, I, B)).astype(np.float32)).to(dev).to(dtype)
    xs, Ws, caches = [], [], []
    inp = x
    for l in range(layers):
        Il = I if l == 0 else H
        W = torch.from_numpy(rng.uniform(-0.2, 0.2, (4 * H, Il + H)).astype(np.float32))
        W = W.to(dev).to(dtype)
        h, cache = L.fwd_cache(inp, W)
        xs.append(inp)
        Ws.append(W)
        caches.append(cache)
        inp = h
    dH = torch.from_numpy(rng.standard_normal((T, H, B)).astype(np.float32)).to(dev)
    return xs, Ws, caches, dH


def sequential(L, xs, Ws, caches, dH, sparsity, kw):
    outs = [None] * len(xs)
    up = dH
    for l in reversed(range(len(xs))):
        if sparsity > 0:
            o = L.bwd_structsparse(xs[l], Ws[l], caches[l], up, sparsity=sparsity,
                                   want_dX=l > 0, **kw)
        else:
            o = L.bwd_dense(xs[l], Ws[l], caches[l], up, want_dX=l > 0)
        outs[l] = o
        up = o.get("dX")
    return outs


GRAPH_SKIP = pytest.mark.skip(reason="recording a stack call into a HIP graph ended in a host "
                              "segmentation fault on the GPU; its capture sequence follows the "
                              "stream-capture rules as modelled on the CPU "
                              "(tests/test_capture_model.py), so the cause is not found and the "
                              "library enqueues stack calls directly")


@pytest.mark.parametrize("graphs", [pytest.param(True, marks=GRAPH_SKIP), False])
@pytest.mark.parametrize("layers,T,B,I,H,sparsity,kw,dx_steps", [
    (2, 9, 20, 40, 64, 0.5, {"P": 4, "R": 8}, 0),
    (3, 12, 64, 96, 128, 0.5, {"P": 4, "R": 8}, 0),
    (3, 12, 64, 96, 128, 0.5, {"P": 4, "R": 8}, 5),    # ragged last chunk
    (2, 8, 128, 64, 64, 0.0, {}, 0),                   # dense
    (2, 7, 64, 32, 64, 0.5, {"kind": 1, "My": 16, "Mx": 4}, 2),  # fine structure
    (4, 16, 32, 48, 96, 0.25, {"P": 4, "R": 8}, 1),    # one step per launch
    (3, 10, 64, 64, 64, 0.5, {"kind": 1, "My": 32, "Mx": 32}, 4),  # 32 x 32 fine blocks
    (1, 6, 32, 40, 64, 0.5, {"P": 4, "R": 8}, 0),      # one layer: the single-layer call
])
def test_stack_matches_sequential(L, graphs, layers, T, B, I, H, sparsity, kw, dx_steps):
    xs, Ws, caches, dH = make_stack(L, layers, T, B, I, H, seed=layers * 10 + T)
    L.graphs_enable(graphs)
    L.set_option("stack_dx_steps", dx_steps)
    try:
        ref = sequential(L, xs, Ws, caches, dH, sparsity, kw)
        for _ in range(2):   # a second call reuses the streams and chunk events
            got = L.bwd_stack(xs, Ws, caches, dH, sparsity=sparsity, **kw)
            torch.cuda.synchronize()
            for l in range(layers):
                assert torch.equal(got["dW"][l], ref[l]["dW"]), ("dW", l)
                assert torch.equal(got["db"][l], ref[l]["db"]), ("db", l)
                if l > 0:
                    assert torch.equal(got["dX"][l], ref[l]["dX"]), ("dX", l)
                if sparsity > 0:
                    assert torch.equal(got["idx"][l], ref[l]["idx"]), ("idx", l)
    finally:
        L.graphs_enable(True)
        L.set_option("stack_dx_steps", 0)


def workload_stack(L, name, layers, T):
    """GPU tensors of the first `layers` layers of a workload (T steps): the
    per-layer inputs (layer l > 0 takes the h_out of the layer below),
    weights and caches, and the top layer's upstream gradient."""
    wl = WORKLOADS[name].truncated(T)
    inp = make_inputs(wl, seed=0)
    dev = torch.device("cuda:0")
    xs, Ws, caches = [], [], []
    x = torch.from_numpy(inp["x"]).to(dev)
    for l in range(layers):
        W = torch.from_numpy(inp["Ws"][l]).to(dev)
        h, cache = L.fwd_cache(x, W)
        xs.append(x)
        Ws.append(W)
        caches.append(cache)
        x = h
    dH = torch.from_numpy(inp["dH_up"]).to(dev)
    return xs, Ws, caches, dH


def test_stack_headline_shape_matches_sequential(L):
    """The benchmark's step call at its layer shape (I = H = 2048, B = 128):
    two layers over T = 26 steps, so each layer's input gradient comes in
    launches of 12, 12 and 2 steps under the cross-layer waits, with the
    two-kernel gate path and 64 x 64 DMA tiles; the bottom layer's input
    gradient too (the benchmark asks for it).  Same bits as the layers'
    calls in turn."""
    xs, Ws, caches, dH = workload_stack(L, "lstm4_enc_h2048_b128_t50_f32", 2, 26)
    kw = {"P": 4, "R": 8}
    ref = sequential(L, xs, Ws, caches, dH, 0.5, kw)
    ref[0] = L.bwd_structsparse(xs[0], Ws[0], caches[0], ref[1]["dX"], sparsity=0.5, **kw)
    got = L.bwd_stack(xs, Ws, caches, dH, sparsity=0.5, want_dX0=True, **kw)
    torch.cuda.synchronize()
    for l in range(2):
        for k in ("dW", "db", "dX", "idx"):
            assert torch.equal(got[k][l], ref[l][k]), (k, l)


def test_stack_headline_shape_oracle(L):
    """The benchmark's step call, the four-layer wavefront stack at the
    4-layer workload's shape with T = 14 (one 12-step and one 2-step input-
    gradient launch per layer), against the oracle: every layer's masks in
    situ (the stack's indices equal those of the layers' calls in turn,
    whose pre-sparsify gate gradients the oracle re-selects bit for bit),
    and every layer's dW, db and dX against the oracle run with those masks
    on the stack's own upstream gradient, to rel. L2 <= 1e-5."""
    layers, T, P, R, S = 4, 14, 4, 8, 4
    xs, Ws, caches, dH = workload_stack(L, "lstm4_enc_h2048_b128_t50_f32", layers, T)
    got = L.bwd_stack(xs, Ws, caches, dH, sparsity=0.5, P=P, R=R, want_dX0=True)
    torch.cuda.synchronize()
    H = Ws[0].shape[0] // 4
    up = dH
    for l in reversed(range(layers)):
        # in situ: the layer's own call (same kernels) with its gate gradients
        o = L.bwd_structsparse(xs[l], Ws[l], caches[l], up, sparsity=0.5, P=P, R=R,
                               want_dbg=True)
        torch.cuda.synchronize()
        assert torch.equal(o["idx"], got["idx"][l]), l
        assert torch.equal(o["dW"], got["dW"][l]), l
        idx = got["idx"][l].cpu().numpy()
        dbg = o["dbg"].double().cpu().numpy()
        keep = np.zeros((T, 4 * H // P), np.uint8)
        for t in range(T):
            k = oracle.select(oracle.scores(dbg[t], P), R, S)
            assert np.array_equal(oracle.kept_index(k), idx[t]), (l, t)
            keep[t] = k
        # gradients against the oracle with the stack's masks
        x_np = xs[l].double().cpu().numpy()
        W_np = Ws[l].double().cpu().numpy()
        gates, c, h = oracle.forward(x_np, W_np)
        ref = oracle.backward(x_np, W_np, gates, c, h, up.double().cpu().numpy(), P=P, R=R, S=S,
                              forced_keep=keep)
        for k in ("dW", "db", "dX"):
            e = rel(got[k][l], ref[k])
            assert e <= 1e-5, (l, k, e)
        up = got["dX"][l]


@pytest.mark.parametrize("struct", [
    {"P": 4, "R": 8},                                  # the benchmark's coarse structure
    {"kind": 1, "My": 8, "Mx": 4},                     # the fine 8 x 4 blocks it also times
    {"kind": 1, "My": 32, "Mx": 32},                   # and the 32 x 32 blocks
])
def test_stack_headline_full_length_sampled(L, struct):
    """The benchmark's timed calls themselves: the four-layer stack at
    I = H = 2048, B = 128, T = 50 (input-gradient launches of 12, 12, 12, 12
    and 2 steps), coarse and fine.  Every layer equals its own call in turn on
    the stack's upstream gradient (dW, db, dX and idx bit for bit); each
    layer's masks at three steps against the oracle's selection; sampled dW
    and dX entries summed in fp64 from the layer's gate gradients, masks and
    inputs (sections 3 and 4: the products run over the kept rows or blocks)."""
    layers, T = 4, 50
    fine = struct.get("kind") == 1
    xs, Ws, caches, dH = workload_stack(L, "lstm4_enc_h2048_b128_t50_f32", layers, T)
    kw = dict(struct)
    if fine:
        kw["kind"] = L.FINE
    got = L.bwd_stack(xs, Ws, caches, dH, sparsity=0.5, want_dX0=True, **kw)
    torch.cuda.synchronize()
    H = Ws[0].shape[0] // 4
    B = dH.shape[2]
    dev = torch.device("cuda:0")
    rng = np.random.default_rng(11)
    n = 32
    up = dH
    for l in reversed(range(layers)):
        I = xs[l].shape[1]
        o = L.bwd_structsparse(xs[l], Ws[l], caches[l], up, sparsity=0.5, want_dbg=True, **kw)
        torch.cuda.synchronize()
        for k in ("dW", "db", "dX", "idx"):
            assert torch.equal(o[k], got[k][l]), (l, k)
        idx = got["idx"][l].cpu().numpy()
        # row mask [T][4H][B] of the kept entries, checked at three steps
        if fine:
            My, Mx = struct["My"], struct["Mx"]
            nb = oracle.fine_blocks(B, My)
            K = int(round(0.5 * nb))
            idx = idx.reshape(T, 4 * H // Mx, nb - K)
            for t in (0, T // 2, T - 1):
                k = oracle.fine_select(oracle.fine_scores(o["dbg"][t].double().cpu().numpy(), Mx, My), K)
                assert np.array_equal(oracle.fine_kept_index(k, K), idx[t]), (l, t)
            keep = np.zeros((T, 4 * H // Mx, nb), np.uint8)
            for t in range(T):
                for sl in range(4 * H // Mx):
                    keep[t, sl, idx[t, sl][idx[t, sl] >= 0]] = 1
            mask = np.repeat(np.repeat(keep, Mx, axis=1), My, axis=2)[:, :, :B]
        else:
            P, R = struct["P"], struct["R"]
            S = int(round(0.5 * R))
            for t in (0, T // 2, T - 1):
                k = oracle.select(oracle.scores(o["dbg"][t].double().cpu().numpy(), P), R, S)
                assert np.array_equal(oracle.kept_index(k), idx[t]), (l, t)
            keep = np.zeros((T, 4 * H // P), np.uint8)
            for t in range(T):
                keep[t, idx[t]] = 1
            mask = np.broadcast_to(np.repeat(keep, P, axis=1)[:, :, None], (T, 4 * H, B))
        _, _, h = L.cache_views(caches[l], T, B, H, "f32")
        rows = rng.integers(0, 4 * H, n)
        cols = rng.integers(0, I + H, n)
        g = o["dbg"].index_select(1, torch.from_numpy(rows).to(dev)).double().cpu().numpy()
        xh = np.empty((T, n, B))
        for j, c in enumerate(cols):
            src = xs[l][:, c, :] if c < I else h[:T, c - I, :]       # h[t] = h_{t-1}
            xh[:, j, :] = src.double().cpu().numpy()
        terms = mask[:, rows, :].astype(np.float64) * g * xh
        gotw = got["dW"][l][torch.from_numpy(rows).to(dev), torch.from_numpy(cols).to(dev)]
        err = np.abs(gotw.double().cpu().numpy() - terms.sum(axis=(0, 2)))
        assert np.all(err <= 2e-5 * np.abs(terms).sum(axis=(0, 2)) + 1e-30), (l, err.max())
        ts, ii, bb = rng.integers(0, T, n), rng.integers(0, I, n), rng.integers(0, B, n)
        Wx = Ws[l][:, torch.from_numpy(ii).to(dev)].double().cpu().numpy()
        for j in range(n):
            t = ts[j]
            tj = (mask[t, :, bb[j]].astype(np.float64) *
                  o["dbg"][t, :, bb[j]].double().cpu().numpy() * Wx[:, j])
            e = abs(got["dX"][l][t, ii[j], bb[j]].item() - tj.sum())
            assert e <= 2e-5 * np.abs(tj).sum() + 1e-30, (l, j, e)
        up = got["dX"][l]


def test_stack_bf16(L):
    xs, Ws, caches, dH = make_stack(L, 2, 6, 64, 64, 128, seed=3, dtype=torch.bfloat16)
    ref = sequential(L, xs, Ws, caches, dH, 0.5, {"P": 4, "R": 8})
    got = L.bwd_stack(xs, Ws, caches, dH, sparsity=0.5)
    torch.cuda.synchronize()
    for l in range(2):
        assert torch.equal(got["dW"][l], ref[l]["dW"])
        assert torch.equal(got["idx"][l], ref[l]["idx"])
