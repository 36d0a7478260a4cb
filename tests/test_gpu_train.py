"""GPU parity of dense-after-sparse training steps (section 5) against the
oracle's training step: a sparse step, then a dense one, on a two-layer
stack; the oracle runs each step from the GPU's weights with the GPU's
masks.  Loss, weight and bias updates to rel. L2 <= 1e-5 (fp32); bf16
storage: gradients to 2e-2 and updated weights within one bf16 rounding."""
import numpy as np
import pytest
import torch

import oracle

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def L():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_1806_00512_amd.lstmss as lstmss
    lstmss.load()
    return lstmss


def rel(a, b):
    a, b = np.asarray(a, np.float64), np.asarray(b, np.float64)
    n = np.linalg.norm(b)
    return float(np.linalg.norm(a - b) / (n if n > 0 else 1.0))


def np64(t):
    return t.detach().float().cpu().numpy().astype(np.float64)


def keep_from_idx(idx, nslices):
    keep = np.zeros((idx.shape[0], nslices), np.uint8)
    for t in range(idx.shape[0]):
        keep[t, idx[t]] = 1
    return keep


@pytest.mark.parametrize("dtype,T,B,I,H", [("f32", 4, 16, 24, 32), ("f32", 3, 20, 40, 72),
                                           ("bf16", 3, 32, 32, 64)])
def test_sparse_then_dense_steps(L, dtype, T, B, I, H):
    from paper_1806_00512_amd.train import StackConfig, StackTrainer
    st = torch.bfloat16 if dtype == "bf16" else torch.float32
    rng = np.random.default_rng(T * 100 + H)
    Ws = [rng.uniform(-0.3, 0.3, (4 * H, (I if l == 0 else H) + H)).astype(np.float32)
          for l in range(2)]
    bs = [rng.uniform(-0.1, 0.1, 4 * H).astype(np.float32) for _ in range(2)]
    x = rng.standard_normal((T, I, B)).astype(np.float32)
    y = (rng.standard_normal((T, H, B)) * 0.5).astype(np.float32)
    if dtype == "bf16":
        Ws = [oracle.round_bf16(w).astype(np.float32) for w in Ws]
        x = oracle.round_bf16(x).astype(np.float32)
    dev = torch.device("cuda:0")
    cfg = StackConfig(layers=2, input_size=I, hidden=H, batch=B, steps=T, dtype=st, lr=0.5,
                      sparsity=0.5, P=4, R=8)
    tr = StackTrainer(cfg, [torch.from_numpy(w).to(dev).to(st) for w in Ws],
                      [torch.from_numpy(b).to(dev) for b in bs])
    xg = torch.from_numpy(x).to(dev).to(st)
    yg = torch.from_numpy(y).to(dev)
    for sparse in (True, False):
        W0 = [np64(w) for w in tr.Ws]
        b0 = [np64(b) for b in tr.bs]
        loss = tr.step(xg, yg, sparse)
        torch.cuda.synchronize()
        fk = None
        if sparse:
            fk = [keep_from_idx(tr.idx[l].cpu().numpy(), 4 * H // 4) for l in range(2)]
        nW, nb, ref_loss, outs = oracle.train_step(x, y, W0, b0, 0.5, sparse, P=4, R=8, S=4,
                                                   bf16=dtype == "bf16", forced_keeps=fk)
        tol = 1e-5 if dtype == "f32" else 2e-2
        assert abs(float(loss.cpu()[0]) - ref_loss) <= tol * abs(ref_loss)
        for l in range(2):
            assert rel(np64(tr.outs[l]["dW"]), outs[l]["dW"]) <= tol
            assert rel(np64(tr.outs[l]["db"]), outs[l]["db"]) <= tol
            if dtype == "f32":
                assert rel(np64(tr.Ws[l]) - W0[l], nW[l] - W0[l]) <= tol
            else:
                assert np.all(np.abs(np64(tr.Ws[l]) - nW[l]) <= 2.0 ** -7 * np.abs(nW[l]) + 1e-6)
            assert rel(np64(tr.bs[l]) - b0[l], nb[l] - b0[l]) <= tol


def test_schedule_and_loss_goes_down(L):
    from paper_1806_00512_amd.train import StackConfig, StackTrainer, dense_after_sparse
    sched = dense_after_sparse(8, 0.75)
    assert sched == [True] * 6 + [False] * 2
    T, B, I, H = 5, 32, 16, 32
    rng = np.random.default_rng(9)
    dev = torch.device("cuda:0")
    Ws = [torch.from_numpy(rng.uniform(-0.2, 0.2, (4 * H, (I if l == 0 else H) + H))
                           .astype(np.float32)).to(dev) for l in range(2)]
    bs = [torch.zeros(4 * H, device=dev) for _ in range(2)]
    x = torch.from_numpy(rng.standard_normal((T, I, B)).astype(np.float32)).to(dev)
    y = torch.from_numpy((rng.standard_normal((T, H, B)) * 0.3).astype(np.float32)).to(dev)
    tr = StackTrainer(StackConfig(layers=2, input_size=I, hidden=H, batch=B, steps=T, lr=0.5),
                      Ws, bs)
    losses = tr.train(x, y, sched).cpu().numpy()
    assert np.all(np.isfinite(losses)) and losses[-1] < losses[0]
