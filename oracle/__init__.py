"""CPU oracle for the structurally sparsified LSTM backward pass (arXiv:1806.00512).

TEST INFRASTRUCTURE ONLY: the slow, obviously correct fp64 definition that the
GPU library is checked against.  Only the test suite, the smoke check and the
benchmark's CPU-baseline leg may import this package.  It shares no code with
the GPU library (``paper_1806_00512_amd``) and does not import it.

The arithmetic lives in ``lstm_oracle.c`` (plain C, fp64, one loop per step of
the method, each citing the passage it follows).  This module only marshals
numpy arrays through ctypes and stacks layers.

Function map (section / table of the paper each one follows):
  forward        LSTM cell forward over T steps (the cache the backward reads;
                 section 4 describes the forward computing the gate activations)
  backward       back-propagation through time with coarse-grained structural
                 sparsifying of the gate gradient dnet (section 3, Fig. 1 caption)
  scores         squared L2 norm of each P-row slice (section 3)
  select         keep R-S of every R slices (section 3; Table 1 for R, S)
  kept_index     offset index array of kept slices (section 3, after Fig. 2)
  kept_rows      K' = P * number of kept slices
  fine_scores    squared L2 norm of each My-column block of each Mx-row slice
                 (section 3, Fig. 2(b))
  fine_select    remove the K lowest blocks of every slice (Table 1 for K)
  fine_kept_index  per-slice offset index of the kept blocks
  backward_fine  back-propagation with the fine-grained structure
  round_bf16     round-to-nearest-even to bfloat16 (storage type of the bf16
                 configuration; not from the paper)
  mse_grad       synthetic regression loss on the top layer's hidden states
                 and its gradient (stands in for the datasets' losses)
  sgd            one SGD update with a fixed learning rate (section 4)
  train_step     forward, loss, backward (sparsified or dense), SGD of a layer
                 stack: one step of dense-after-sparse training (section 5)
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "lstm_oracle.c")
_LIB_PATH = os.path.join(_HERE, "liblstm_oracle.so")
_lib = None


def build_library(openmp: bool = True) -> str:
    """Compile lstm_oracle.c into liblstm_oracle.so (gcc, fp64, no fast-math)."""
    cmd = ["gcc", "-O2", "-ffp-contract=off", "-fno-fast-math", "-fPIC", "-shared"]
    if openmp:
        cmd.append("-fopenmp")
    tmp = _LIB_PATH + ".tmp%d" % os.getpid()
    cmd += ["-o", tmp, _SRC, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        build_library()
    lib = ctypes.CDLL(_LIB_PATH)
    P = ctypes.c_void_p
    i = ctypes.c_int
    L = ctypes.c_long
    lib.oracle_forward.argtypes = [i, i, i, i, P, P, P, P, P, i, P, P, P]
    lib.oracle_forward.restype = i
    lib.oracle_scores.argtypes = [L, i, i, P, P]
    lib.oracle_scores.restype = i
    lib.oracle_select.argtypes = [L, i, i, P, P]
    lib.oracle_select.restype = i
    lib.oracle_kept_index.argtypes = [L, P, P]
    lib.oracle_kept_index.restype = L
    lib.oracle_kept_rows.argtypes = [L, i, i, i]
    lib.oracle_kept_rows.restype = L
    lib.oracle_removed_in_region.argtypes = [L, i, i]
    lib.oracle_removed_in_region.restype = L
    lib.oracle_threads.restype = i
    lib.oracle_set_threads.argtypes = [i]
    lib.oracle_set_threads.restype = None
    lib.oracle_round_bf16.argtypes = [ctypes.c_double]
    lib.oracle_round_bf16.restype = ctypes.c_double
    lib.oracle_backward.argtypes = [i, i, i, i, P, P, P, P, P, P, P, P, i, i, i, i, P,
                                    P, P, P, P, P, P, P, P]
    lib.oracle_backward.restype = i
    lib.oracle_fine_blocks.argtypes = [i, i]
    lib.oracle_fine_blocks.restype = L
    lib.oracle_fine_scores.argtypes = [L, i, i, i, P, P]
    lib.oracle_fine_scores.restype = i
    lib.oracle_fine_select.argtypes = [L, L, i, P, P]
    lib.oracle_fine_select.restype = i
    lib.oracle_fine_kept_index.argtypes = [L, L, i, P, P]
    lib.oracle_fine_kept_index.restype = None
    lib.oracle_backward_fine.argtypes = [i, i, i, i, P, P, P, P, P, P, P, P, i, i, i, i, P,
                                         P, P, P, P, P, P, P, P]
    lib.oracle_backward_fine.restype = i
    _lib = lib
    return lib


def _f64(a):
    if a is None:
        return None
    return np.ascontiguousarray(a, dtype=np.float64)


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _check(rc, what):
    if rc != 0:
        raise ValueError("oracle %s failed with code %d" % (what, rc))


def round_bf16(a) -> np.ndarray:
    """Element-wise round-to-nearest-even to bfloat16, returned as float64."""
    lib = _load()
    a = np.asarray(a, dtype=np.float64)
    f = np.vectorize(lib.oracle_round_bf16, otypes=[np.float64])
    return f(a) if a.size else a.copy()


def forward(x, W, b=None, h0=None, c0=None, bf16=False):
    """One layer forward.  x [T][I][B], W [4H][I+H] -> (gates, c, h)."""
    lib = _load()
    x, W, b, h0, c0 = map(_f64, (x, W, b, h0, c0))
    T, I, B = x.shape
    G, K = W.shape
    H = G // 4
    assert K == I + H and G == 4 * H
    gates = np.empty((T, G, B))
    c = np.empty((T + 1, H, B))
    h = np.empty((T + 1, H, B))
    rc = lib.oracle_forward(T, B, I, H, _ptr(x), _ptr(W), _ptr(b), _ptr(h0), _ptr(c0),
                            int(bool(bf16)), _ptr(gates), _ptr(c), _ptr(h))
    _check(rc, "forward")
    return gates, c, h


def threads() -> int:
    """Threads the oracle's parallel loops use."""
    return int(_load().oracle_threads())


def set_threads(n: int) -> None:
    """Threads of the parallel loops (results do not depend on it)."""
    _load().oracle_set_threads(int(n))


def kept_rows(rows: int, P: int, R: int, S: int) -> int:
    return int(_load().oracle_kept_rows(rows, P, R, S))


def removed_in_region(r: int, R: int, S: int) -> int:
    return int(_load().oracle_removed_in_region(r, R, S))


def scores(dG, P: int) -> np.ndarray:
    """Squared L2 norm of each P-row slice of dG [rows][B], fixed fp64 order."""
    lib = _load()
    dG = _f64(dG)
    rows, B = dG.shape
    out = np.empty(rows // P)
    _check(lib.oracle_scores(rows, B, P, _ptr(dG), _ptr(out)), "scores")
    return out


def select(sc, R: int, S: int) -> np.ndarray:
    """Keep mask (uint8) over slices given their scores."""
    lib = _load()
    sc = _f64(sc)
    keep = np.empty(sc.shape[0], dtype=np.uint8)
    _check(lib.oracle_select(sc.shape[0], R, S, _ptr(sc), _ptr(keep)), "select")
    return keep


def kept_index(keep) -> np.ndarray:
    keep = np.ascontiguousarray(keep, dtype=np.uint8)
    idx = np.empty(keep.shape[0], dtype=np.int32)
    n = _load().oracle_kept_index(keep.shape[0], _ptr(keep), _ptr(idx))
    return idx[:n].copy()


def fine_blocks(B: int, My: int) -> int:
    """Blocks of My batch columns per slice (the last one may be narrower)."""
    return int(_load().oracle_fine_blocks(B, My))


def fine_scores(dG, Mx: int, My: int) -> np.ndarray:
    """[rows/Mx][nb] squared L2 norms of the My-column blocks of each slice."""
    lib = _load()
    dG = _f64(dG)
    rows, B = dG.shape
    out = np.empty((rows // Mx, fine_blocks(B, My)))
    _check(lib.oracle_fine_scores(rows, B, Mx, My, _ptr(dG), _ptr(out)), "fine_scores")
    return out


def fine_select(sc, K: int) -> np.ndarray:
    """Keep mask [nslices][nb] (uint8): the K lowest blocks of each slice removed."""
    lib = _load()
    sc = _f64(sc)
    keep = np.empty(sc.shape, dtype=np.uint8)
    _check(lib.oracle_fine_select(sc.shape[0], sc.shape[1], K, _ptr(sc), _ptr(keep)),
           "fine_select")
    return keep


def fine_kept_index(keep, K: int) -> np.ndarray:
    """Per-slice ascending kept block indices [nslices][nb - K] (-1 pads)."""
    keep = np.ascontiguousarray(keep, dtype=np.uint8)
    ns, nb = keep.shape
    out = np.empty((ns, nb - K), dtype=np.int32)
    _load().oracle_fine_kept_index(ns, nb, K, _ptr(keep), _ptr(out))
    return out


def backward_fine(x, W, gates, c, h, dH_up, dhT=None, dcT=None, Mx=4, My=8, K=1, bf16=False,
                  forced_keep=None, want_dX=True, want_dG=False):
    """One layer backward with the fine-grained structure.

    Returns the dict of ``backward`` with keep [T][4H/Mx][nb] (uint8) and
    idx [T][4H/Mx][nb - K] (int32 kept block indices per slice)."""
    lib = _load()
    x, W, gates, c, h, dH_up, dhT, dcT = map(_f64, (x, W, gates, c, h, dH_up, dhT, dcT))
    T, I, B = x.shape
    G, Kc = W.shape
    H = G // 4
    nsl = G // Mx
    nb = fine_blocks(B, My)
    out = {
        "dX": np.empty((T, I, B)) if want_dX else None,
        "dW": np.empty((G, Kc)),
        "db": np.empty(G),
        "dh0": np.empty((H, B)),
        "dc0": np.empty((H, B)),
        "keep": np.empty((T, nsl, nb), dtype=np.uint8),
        "idx": np.empty((T, nsl, nb - K), dtype=np.int32),
        "dG": np.empty((T, G, B)) if want_dG else None,
    }
    fk = None if forced_keep is None else np.ascontiguousarray(forced_keep, dtype=np.uint8)
    if fk is not None:
        assert fk.shape == (T, nsl, nb)
    rc = lib.oracle_backward_fine(T, B, I, H, _ptr(x), _ptr(W), _ptr(gates), _ptr(c), _ptr(h),
                                  _ptr(dH_up), _ptr(dhT), _ptr(dcT), Mx, My, K, int(bool(bf16)),
                                  _ptr(fk), _ptr(out["dX"]), _ptr(out["dW"]), _ptr(out["db"]),
                                  _ptr(out["dh0"]), _ptr(out["dc0"]), _ptr(out["keep"]),
                                  _ptr(out["idx"]), _ptr(out["dG"]))
    _check(rc, "backward_fine")
    return out


def backward(x, W, gates, c, h, dH_up, dhT=None, dcT=None, P=4, R=8, S=4, bf16=False,
             forced_keep=None, want_dX=True, want_dG=False):
    """One layer backward through time.

    Returns a dict with dX [T][I][B] (or None), dW [4H][I+H], db [4H],
    dh0, dc0 [H][B], keep [T][4H/P] (uint8), idx [T][K'/P] (int32) and,
    when want_dG, dG [T][4H][B] before sparsifying.
    """
    lib = _load()
    x, W, gates, c, h, dH_up, dhT, dcT = map(_f64, (x, W, gates, c, h, dH_up, dhT, dcT))
    T, I, B = x.shape
    G, K = W.shape
    H = G // 4
    nsl = G // P
    ks = kept_rows(G, P, R, S) // P
    out = {
        "dX": np.empty((T, I, B)) if want_dX else None,
        "dW": np.empty((G, K)),
        "db": np.empty(G),
        "dh0": np.empty((H, B)),
        "dc0": np.empty((H, B)),
        "keep": np.empty((T, nsl), dtype=np.uint8),
        "idx": np.empty((T, ks), dtype=np.int32),
        "dG": np.empty((T, G, B)) if want_dG else None,
    }
    fk = None if forced_keep is None else np.ascontiguousarray(forced_keep, dtype=np.uint8)
    if fk is not None:
        assert fk.shape == (T, nsl)
    rc = lib.oracle_backward(T, B, I, H, _ptr(x), _ptr(W), _ptr(gates), _ptr(c), _ptr(h),
                             _ptr(dH_up), _ptr(dhT), _ptr(dcT), P, R, S, int(bool(bf16)),
                             _ptr(fk), _ptr(out["dX"]), _ptr(out["dW"]), _ptr(out["db"]),
                             _ptr(out["dh0"]), _ptr(out["dc0"]), _ptr(out["keep"]),
                             _ptr(out["idx"]), _ptr(out["dG"]))
    _check(rc, "backward")
    return out


def stack_forward(x, Ws, bs=None, bf16=False):
    """Multi-layer forward: layer l+1's input is layer l's h[1:]."""
    caches = []
    inp = x
    for li, W in enumerate(Ws):
        b = None if bs is None else bs[li]
        gates, c, h = forward(inp, W, b, bf16=bf16)
        caches.append({"x": np.asarray(inp, dtype=np.float64), "W": W, "gates": gates,
                       "c": c, "h": h})
        inp = h[1:]
    return caches


def stack_backward(caches, dH_up, P=4, R=8, S=4, bf16=False, forced_keeps=None, want_dG=False):
    """Multi-layer backward, top layer first; layer l's dX is layer l-1's dH_up."""
    outs = [None] * len(caches)
    up = dH_up
    for li in reversed(range(len(caches))):
        cc = caches[li]
        fk = None if forced_keeps is None else forced_keeps[li]
        o = backward(cc["x"], cc["W"], cc["gates"], cc["c"], cc["h"], up, P=P, R=R, S=S,
                     bf16=bf16, forced_keep=fk, want_dX=True, want_dG=want_dG)
        outs[li] = o
        up = o["dX"]
    return outs


def mse_grad(h, y):
    """L = (1 / 2B) * sum of (h - y)^2 over [T][H][B] and dL/dh = (h - y) / B.

    A synthetic loss on the top layer's hidden states: the paper's losses come
    from datasets that are not used here; any differentiable loss exercises
    the same backward pass."""
    h, y = _f64(h), _f64(y)
    B = h.shape[-1]
    dif = h - y
    return dif / B, 0.5 * float(np.sum(dif * dif)) / B


def sgd(W, dW, lr, bf16=False):
    """W - lr * dW (section 4: plain SGD with a fixed learning rate), rounded to
    bfloat16 when the weights are stored in it."""
    out = _f64(W) - float(lr) * _f64(dW)
    return round_bf16(out) if bf16 else out


def train_step(x, y, Ws, bs, lr, sparse, P=4, R=8, S=4, bf16=False, forced_keeps=None):
    """One training step of a layer stack (zero initial state): forward, loss
    gradient at the top, backward through every layer top first (coarse
    sparsifying when ``sparse``, else dense), SGD on every W and b.

    Returns (new Ws, new bs, loss, per-layer backward outputs)."""
    caches = stack_forward(x, Ws, bs, bf16=bf16)
    dH, loss = mse_grad(caches[-1]["h"][1:], y)
    if sparse:
        outs = stack_backward(caches, dH, P=P, R=R, S=S, bf16=bf16, forced_keeps=forced_keeps)
    else:
        outs = stack_backward(caches, dH, P=4, R=8, S=0, bf16=bf16)
    new_W = [sgd(W, o["dW"], lr, bf16) for W, o in zip(Ws, outs)]
    new_b = [sgd(b, o["db"], lr) for b, o in zip(bs, outs)]
    return new_W, new_b, loss, outs
