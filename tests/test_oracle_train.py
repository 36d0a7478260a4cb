"""Pins of the oracle's training-step pieces (loss gradient, SGD, one step of
a layer stack) against finite differences and closed forms."""
import numpy as np
import pytest

import oracle


def test_mse_grad_closed_form():
    T, H, B = 3, 4, 5
    y = np.zeros((T, H, B))
    h = np.ones((T, H, B))
    dH, L = oracle.mse_grad(h, y)
    assert L == pytest.approx(T * H / 2.0, rel=1e-15)   # (1/2B) * T*H*B * 1^2
    assert np.all(dH == 1.0 / B)
    dH, L = oracle.mse_grad(y, y)
    assert L == 0.0 and np.all(dH == 0.0)


def test_mse_grad_finite_differences():
    rng = np.random.default_rng(1)
    h = rng.standard_normal((2, 3, 4))
    y = rng.standard_normal((2, 3, 4))
    dH, _ = oracle.mse_grad(h, y)
    eps = 1e-6
    for i in [(0, 0, 0), (1, 2, 3), (0, 1, 2)]:
        hp, hm = h.copy(), h.copy()
        hp[i] += eps
        hm[i] -= eps
        fd = (oracle.mse_grad(hp, y)[1] - oracle.mse_grad(hm, y)[1]) / (2 * eps)
        assert fd == pytest.approx(dH[i], rel=1e-7, abs=1e-10)


def test_sgd_quadratic_and_bf16_rounding():
    rng = np.random.default_rng(2)
    Wstar = rng.standard_normal((4, 6))
    W = rng.standard_normal((4, 6))
    # f(W) = |W - W*|^2 / 2 has gradient W - W*: one step of lr 1 lands on W*
    assert np.allclose(oracle.sgd(W, W - Wstar, 1.0), Wstar, rtol=0, atol=1e-15)
    assert np.allclose(oracle.sgd(W, W - Wstar, 0.5), (W + Wstar) / 2, rtol=0, atol=1e-15)
    # bf16 storage: 1 + 2^-9 is below half an ulp (2^-8) of 1 -> 1; 1 + 3*2^-8
    # is a tie between 1 + 2^-7 (odd mantissa) and 1 + 2^-6 (even) -> 1 + 2^-6
    one = np.ones((1, 2))
    out = oracle.sgd(one, np.array([[-2.0 ** -9, -3 * 2.0 ** -8]]), 1.0, bf16=True)
    assert out[0, 0] == 1.0 and out[0, 1] == 1.0 + 2.0 ** -6


def _stack(seed, T=3, B=2, I=3, H=2, layers=2):
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((T, I, B))
    y = rng.standard_normal((T, H, B)) * 0.5
    Ws = [rng.uniform(-0.5, 0.5, (4 * H, (I if l == 0 else H) + H)) for l in range(layers)]
    bs = [rng.uniform(-0.2, 0.2, 4 * H) for _ in range(layers)]
    return x, y, Ws, bs


def _loss(x, y, Ws, bs):
    caches = oracle.stack_forward(x, Ws, bs)
    return oracle.mse_grad(caches[-1]["h"][1:], y)[1]


def test_dense_train_step_gradient_is_the_loss_gradient():
    """The dense step's dW, db of every layer (loss gradient at the top, dX
    chained down the stack) match central differences of the stack's loss."""
    x, y, Ws, bs = _stack(3)
    lr = 0.1
    nW, nb, L, outs = oracle.train_step(x, y, Ws, bs, lr, sparse=False)
    assert L == pytest.approx(_loss(x, y, Ws, bs), rel=1e-14)
    eps = 1e-6
    for l in range(len(Ws)):
        for (i, j) in [(0, 0), (3, 1), (7, 2)]:
            Wp = [w.copy() for w in Ws]
            Wm = [w.copy() for w in Ws]
            Wp[l][i, j] += eps
            Wm[l][i, j] -= eps
            fd = (_loss(x, y, Wp, bs) - _loss(x, y, Wm, bs)) / (2 * eps)
            assert fd == pytest.approx(outs[l]["dW"][i, j], rel=1e-6, abs=1e-10)
        for i in (1, 6):
            bp = [b.copy() for b in bs]
            bm = [b.copy() for b in bs]
            bp[l][i] += eps
            bm[l][i] -= eps
            fd = (_loss(x, y, Ws, bp) - _loss(x, y, Ws, bm)) / (2 * eps)
            assert fd == pytest.approx(outs[l]["db"][i], rel=1e-6, abs=1e-10)
        assert np.allclose(nW[l], Ws[l] - lr * outs[l]["dW"], rtol=0, atol=1e-15)
        assert np.allclose(nb[l], bs[l] - lr * outs[l]["db"], rtol=0, atol=1e-15)


def test_sparse_step_without_removal_equals_dense():
    x, y, Ws, bs = _stack(4, T=3, B=3, I=4, H=4)
    a = oracle.train_step(x, y, Ws, bs, 0.3, sparse=False)
    b = oracle.train_step(x, y, Ws, bs, 0.3, sparse=True, P=4, R=4, S=0)
    for l in range(2):
        assert np.array_equal(a[0][l], b[0][l]) and np.array_equal(a[1][l], b[1][l])


def test_sparse_step_updates_only_kept_rows():
    """With coarse sparsifying the removed slices' rows of dW and db are zero
    at every step where they are removed; rows removed at every step keep W."""
    x, y, Ws, bs = _stack(5, T=1, B=3, I=4, H=8)
    nW, nb, _, outs = oracle.train_step(x, y, Ws, bs, 0.5, sparse=True, P=4, R=8, S=4)
    for l in range(2):
        keep = outs[l]["keep"][0]
        assert keep.sum() == 4
        for j in np.flatnonzero(keep == 0):
            rows = slice(4 * j, 4 * j + 4)
            assert np.array_equal(nW[l][rows], Ws[l][rows])
            assert np.array_equal(nb[l][rows], bs[l][rows])
