"""Python binding of liblstmss (ctypes): torch tensors in, device pointers out.

Argument marshalling only: every step of the forward and backward passes runs
in the HIP kernels of liblstmss.so.  torch provides device memory and the
current stream.  The entry points mirror include/lstmss.h:

  fwd_cache              -> lstm_fwd_cache
  bwd_dense              -> lstm_bwd_dense
  bwd_structsparse       -> lstm_bwd_structsparse
  select_compact         -> lstmss_select_compact
  cache_bytes / kept_rows / index_entries / workspace_bytes -> the size queries

Loading fails loudly (RuntimeError) when liblstmss.so has not been built;
there is no fallback implementation.
"""
from __future__ import annotations

import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "liblstmss.so")

F32, BF16 = 0, 1
COARSE, FINE = 0, 1
ERR = {0: "ok", -1: "invalid argument", -2: "unsupported", -3: "workspace too small",
       -4: "HIP runtime error"}

# Exported symbols of include/lstmss.h
SYMBOLS = ("lstmss_version", "lstmss_strerror", "lstmss_last_error", "lstmss_cache_bytes",
           "lstmss_kept_rows", "lstmss_bwd_info", "lstmss_index_entries", "lstmss_workspace_bytes",
           "lstmss_fwd_workspace_bytes", "lstmss_sgd_update", "lstmss_mse_grad",
           "lstmss_stack_workspace_bytes", "lstm_bwd_stack", "lstmss_time_reverse",
           "lstmss_bidir_join", "lstmss_bidir_workspace_bytes", "lstm_bwd_bidir",
           "lstm_fwd_cache", "lstm_bwd_dense",
           "lstm_bwd_structsparse", "lstmss_select_workspace_bytes", "lstmss_select_compact",
           "lstmss_select_compact_noalloc", "lstmss_set_option",
           "lstmss_timing_enable", "lstmss_timing_read", "lstmss_timing_reset")
KERNEL_KINDS = {"gates_select_compact": 0, "data_grad_gemm": 1, "weight_grad_gemm": 2, "aux": 3,
                "forward_step": 4}


class Dims(ctypes.Structure):
    _fields_ = [("T", ctypes.c_int32), ("B", ctypes.c_int32), ("I", ctypes.c_int32),
                ("H", ctypes.c_int32), ("dtype", ctypes.c_int32)]


class Structure(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int32), ("P", ctypes.c_int32), ("R", ctypes.c_int32),
                ("My", ctypes.c_int32), ("Mx", ctypes.c_int32)]


class LstmssError(RuntimeError):
    def __init__(self, code, what, detail):
        super().__init__("%s: %s (%d): %s" % (what, ERR.get(code, "?"), code, detail))
        self.code = code


_lib = None


def load():
    """Load liblstmss.so (built in-tree by __graft_entry__.build())."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError("liblstmss.so is not built (%s); run __graft_entry__.build()" % LIB_PATH)
    lib = ctypes.CDLL(LIB_PATH)
    vp, i32, i64, f = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_float
    pd, ps = ctypes.POINTER(Dims), ctypes.POINTER(Structure)
    lib.lstmss_version.restype = i32
    lib.lstmss_strerror.argtypes = [i32]
    lib.lstmss_strerror.restype = ctypes.c_char_p
    lib.lstmss_last_error.restype = ctypes.c_char_p
    lib.lstmss_cache_bytes.argtypes = [pd]
    lib.lstmss_cache_bytes.restype = i64
    lib.lstmss_kept_rows.argtypes = [pd, f, ps]
    lib.lstmss_kept_rows.restype = i64
    lib.lstmss_bwd_info.argtypes = [pd, f, ps, ctypes.POINTER(ctypes.c_int32)]
    lib.lstmss_bwd_info.restype = ctypes.c_int32
    lib.lstmss_index_entries.argtypes = [pd, f, ps]
    lib.lstmss_index_entries.restype = i64
    lib.lstmss_workspace_bytes.argtypes = [pd, f, ps]
    lib.lstmss_workspace_bytes.restype = i64
    lib.lstmss_fwd_workspace_bytes.argtypes = [pd]
    lib.lstmss_fwd_workspace_bytes.restype = i64
    lib.lstm_fwd_cache.argtypes = [pd, vp, vp, vp, vp, vp, vp, vp, vp, ctypes.c_size_t, vp]
    lib.lstm_fwd_cache.restype = i32
    lib.lstmss_sgd_update.argtypes = [pd, vp, vp, vp, vp, f, vp]
    lib.lstmss_sgd_update.restype = i32
    lib.lstmss_mse_grad.argtypes = [pd, vp, vp, vp, vp, vp]
    lib.lstmss_mse_grad.restype = i32
    lib.lstmss_stack_workspace_bytes.argtypes = [i32, pd, f, ps]
    lib.lstmss_stack_workspace_bytes.restype = i64
    lib.lstm_bwd_stack.argtypes = [i32, pd, f, ps, vp, vp, vp, vp, vp, vp, vp, vp, vp,
                                   ctypes.c_size_t, vp]
    lib.lstm_bwd_stack.restype = i32
    lib.lstmss_time_reverse.argtypes = [i32, i64, vp, vp, vp]
    lib.lstmss_time_reverse.restype = i32
    lib.lstmss_bidir_join.argtypes = [pd, vp, vp, vp, vp]
    lib.lstmss_bidir_join.restype = i32
    lib.lstmss_bidir_workspace_bytes.argtypes = [pd, f, ps]
    lib.lstmss_bidir_workspace_bytes.restype = i64
    lib.lstm_bwd_bidir.argtypes = [pd, f, ps] + [vp] * 15 + [ctypes.c_size_t, vp]
    lib.lstm_bwd_bidir.restype = i32
    lib.lstm_bwd_dense.argtypes = [pd, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp,
                                   ctypes.c_size_t, vp]
    lib.lstm_bwd_dense.restype = i32
    lib.lstm_bwd_structsparse.argtypes = [pd, f, ps, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp,
                                          vp, vp, vp, ctypes.c_size_t, vp]
    lib.lstm_bwd_structsparse.restype = i32
    lib.lstmss_select_workspace_bytes.argtypes = [pd, f, ps]
    lib.lstmss_select_workspace_bytes.restype = i64
    lib.lstmss_select_compact.argtypes = [pd, f, ps, vp, vp, vp, vp, vp, ctypes.c_size_t, vp]
    lib.lstmss_select_compact.restype = i32
    lib.lstmss_select_compact_noalloc.argtypes = [pd, f, ps, vp, vp, vp, vp, vp]
    lib.lstmss_select_compact_noalloc.restype = i32
    lib.lstmss_set_option.argtypes = [i32, i32]
    lib.lstmss_set_option.restype = i32
    lib.lstmss_timing_enable.argtypes = [i32]
    lib.lstmss_timing_enable.restype = i32
    lib.lstmss_timing_read.argtypes = [i32, ctypes.POINTER(ctypes.c_double),
                                       ctypes.POINTER(ctypes.c_int64)]
    lib.lstmss_timing_read.restype = i32
    lib.lstmss_timing_reset.restype = i32
    _lib = lib
    return lib


def _check(code, what):
    if code != 0:
        detail = load().lstmss_last_error().decode()
        raise LstmssError(code, what, detail)


def _dt(dtype):
    if dtype in (torch.float32, "f32", F32):
        return F32
    if dtype in (torch.bfloat16, "bf16", BF16):
        return BF16
    raise ValueError("unsupported storage dtype %r" % (dtype,))


def torch_dtype(dt):
    return torch.bfloat16 if _dt(dt) == BF16 else torch.float32


def dims(T, B, I, H, dtype=F32) -> Dims:
    return Dims(int(T), int(B), int(I), int(H), _dt(dtype))


def structure(P=4, R=8, kind=COARSE, My=0, Mx=0) -> Structure:
    """COARSE uses P, R; FINE uses My (block width), Mx (rows per slice)."""
    return Structure(int(kind), int(P), int(R), int(My), int(Mx))


def _ptr(t, dtype=None, shape=None, name="tensor"):
    if t is None:
        return None
    if not isinstance(t, torch.Tensor):
        raise TypeError("%s must be a torch tensor" % name)
    if t.device.type != "cuda":
        raise ValueError("%s must live on the GPU" % name)
    if not t.is_contiguous():
        raise ValueError("%s must be contiguous" % name)
    if dtype is not None and t.dtype != dtype:
        raise ValueError("%s has dtype %s, expected %s" % (name, t.dtype, dtype))
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError("%s has shape %s, expected %s" % (name, tuple(t.shape), tuple(shape)))
    return ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def cache_bytes(d: Dims) -> int:
    n = load().lstmss_cache_bytes(ctypes.byref(d))
    _check(0 if n >= 0 else int(n), "lstmss_cache_bytes")
    return int(n)


def kept_rows(d: Dims, sparsity: float, s: Structure) -> int:
    n = load().lstmss_kept_rows(ctypes.byref(d), float(sparsity), ctypes.byref(s))
    _check(0 if n >= 0 else int(n), "lstmss_kept_rows")
    return int(n)


INFO_SPLIT_GATES = 1
INFO_SELECT_IN_PRODUCT = 2


def bwd_info(d: Dims, sparsity: float, s: Structure) -> dict:
    """How the backward runs the gate path for these arguments (current
    options): {"split_gates": bool, "select_in_product": bool}."""
    f = ctypes.c_int32(0)
    _check(load().lstmss_bwd_info(ctypes.byref(d), float(sparsity), ctypes.byref(s),
                                  ctypes.byref(f)), "lstmss_bwd_info")
    return {"split_gates": bool(f.value & INFO_SPLIT_GATES),
            "select_in_product": bool(f.value & INFO_SELECT_IN_PRODUCT)}


def index_entries(d: Dims, sparsity: float, s: Structure) -> int:
    n = load().lstmss_index_entries(ctypes.byref(d), float(sparsity), ctypes.byref(s))
    _check(0 if n >= 0 else int(n), "lstmss_index_entries")
    return int(n)


def workspace_bytes(d: Dims, sparsity: float = 0.0, s: Structure | None = None) -> int:
    n = load().lstmss_workspace_bytes(ctypes.byref(d), float(sparsity),
                                      ctypes.byref(s) if s is not None else None)
    _check(0 if n >= 0 else int(n), "lstmss_workspace_bytes")
    return int(n)


def select_workspace_bytes(d: Dims, sparsity: float, s: Structure) -> int:
    """Scratch of lstmss_select_compact (0 unless the shape takes the
    two-kernel path of the backward pass)."""
    n = load().lstmss_select_workspace_bytes(ctypes.byref(d), float(sparsity), ctypes.byref(s))
    _check(0 if n >= 0 else int(n), "lstmss_select_workspace_bytes")
    return int(n)


def fwd_workspace_bytes(d: Dims) -> int:
    n = load().lstmss_fwd_workspace_bytes(ctypes.byref(d))
    _check(0 if n >= 0 else int(n), "lstmss_fwd_workspace_bytes")
    return int(n)


def fwd_cache(x, W, b=None, h0=None, c0=None, h_out=None, cache=None, stream=None, ws=None,
              batched=True):
    """x [T][I][B], W [4H][I+H] (fp32 or bf16) -> (h_out [T][H][B], cache bytes).

    batched: the input projection of all steps as one product plus split
    recurrent products (needs a workspace, allocated here unless ws is
    given); False: the fused per-step kernel without scratch."""
    T, I, B = x.shape
    H = W.shape[0] // 4
    st = x.dtype
    d = dims(T, B, I, H, st)
    if cache is None:
        cache = torch.empty(cache_bytes(d), dtype=torch.uint8, device=x.device)
    if h_out is None:
        h_out = torch.empty((T, H, B), dtype=st, device=x.device)
    if batched and ws is None:
        ws = torch.empty(fwd_workspace_bytes(d), dtype=torch.uint8, device=x.device)
    if not batched:
        ws = None
    rc = load().lstm_fwd_cache(ctypes.byref(d), _ptr(x, st, name="x"),
                               _ptr(W, st, (4 * H, I + H), "W"),
                               _ptr(b, torch.float32, (4 * H,), "b"),
                               _ptr(h0, torch.float32, (H, B), "h0"),
                               _ptr(c0, torch.float32, (H, B), "c0"),
                               _ptr(h_out, st, (T, H, B), "h_out"),
                               _ptr(cache, torch.uint8, name="cache"),
                               _ptr(ws, torch.uint8, name="ws"), 0 if ws is None else ws.numel(),
                               _stream(stream))
    _check(rc, "lstm_fwd_cache")
    return h_out, cache


LOSS_SLOTS = 1025


def sgd_update(W, b, dW, db, lr, I, stream=None):
    """In place: W -= lr dW (storage type of W), b -= lr db (b may be None)."""
    G, K = W.shape
    H = G // 4
    d = dims(1, 1, I, H, W.dtype)
    f32 = torch.float32
    rc = load().lstmss_sgd_update(ctypes.byref(d), _ptr(W, W.dtype, (G, I + H), "W"),
                                  _ptr(b, f32, (G,), "b"), _ptr(dW, f32, (G, I + H), "dW"),
                                  _ptr(db, f32, (G,), "db"), float(lr), _stream(stream))
    _check(rc, "lstmss_sgd_update")


def mse_grad(h, y, dH=None, loss=None, stream=None):
    """dH = (h - y) / B and the loss (1/2B) sum (h - y)^2 (fp64 device array of
    LOSS_SLOTS, the loss in its last slot).  Returns (dH, loss)."""
    T, H, B = h.shape
    d = dims(T, B, 1, H, h.dtype)
    if dH is None:
        dH = torch.empty((T, H, B), dtype=torch.float32, device=h.device)
    if loss is None:
        loss = torch.empty(LOSS_SLOTS, dtype=torch.float64, device=h.device)
    rc = load().lstmss_mse_grad(ctypes.byref(d), _ptr(h, h.dtype, name="h"),
                                _ptr(y, torch.float32, (T, H, B), "y"),
                                _ptr(dH, torch.float32, (T, H, B), "dH"),
                                _ptr(loss, torch.float64, (LOSS_SLOTS,), "loss"), _stream(stream))
    _check(rc, "lstmss_mse_grad")
    return dH, loss


def _ptr_array(ts, name, dtype=None):
    """ctypes array of device pointers (None entries -> NULL)."""
    arr = (ctypes.c_void_p * len(ts))()
    for i, t in enumerate(ts):
        p = _ptr(t, dtype, name="%s[%d]" % (name, i))
        arr[i] = None if p is None else p.value
    return arr


def stack_workspace_bytes(ds, sparsity: float = 0.0, s: Structure | None = None) -> int:
    """Workspace of lstm_bwd_stack for the per-layer dims ds (list of Dims)."""
    arr = (Dims * len(ds))(*ds)
    n = load().lstmss_stack_workspace_bytes(len(ds), arr, float(sparsity),
                                            ctypes.byref(s) if s is not None else None)
    _check(0 if n >= 0 else int(n), "lstmss_stack_workspace_bytes")
    return int(n)


def bwd_stack(xs, Ws, caches, dH_top, sparsity=0.5, P=4, R=8, kind=COARSE, My=0, Mx=0,
              dXs=None, dWs=None, dbs=None, idxs=None, ws=None, want_dX0=False, stream=None):
    """Wavefront backward of a layer stack (layer 0 at the bottom): per-layer
    lists xs [T][I_l][B], Ws, caches; dH_top [T][H][B].  sparsity 0 = dense.
    Returns dict(dX, dW, db, idx) of per-layer lists."""
    n = len(xs)
    T, _, B = xs[0].shape
    st = xs[0].dtype
    dev = xs[0].device
    f32 = torch.float32
    ds = (Dims * n)()
    for l in range(n):
        ds[l] = dims(T, B, xs[l].shape[1], Ws[l].shape[0] // 4, st)
    s = structure(P, R, kind, My, Mx) if sparsity > 0 else None
    sp = float(sparsity)
    if dWs is None:
        dWs = [torch.empty(tuple(W.shape), dtype=f32, device=dev) for W in Ws]
    if dbs is None:
        dbs = [torch.empty(W.shape[0], dtype=f32, device=dev) for W in Ws]
    if dXs is None:
        dXs = [torch.empty(tuple(x.shape), dtype=f32, device=dev) if (l > 0 or want_dX0) else None
               for l, x in enumerate(xs)]
    if idxs is None and s is not None:
        idxs = [torch.empty((T, index_entries(ds[l], sp, s)), dtype=torch.int32, device=dev)
                for l in range(n)]
    if ws is None:
        ws = torch.empty(stack_workspace_bytes(list(ds), sp, s), dtype=torch.uint8, device=dev)
    rc = load().lstm_bwd_stack(
        n, ds, sp, ctypes.byref(s) if s else None, _ptr_array(xs, "x", st),
        _ptr_array(Ws, "W", st), _ptr_array(caches, "cache", torch.uint8),
        _ptr(dH_top, f32, name="dH_top"), _ptr_array(dXs, "dX", f32), _ptr_array(dWs, "dW", f32),
        _ptr_array(dbs, "db", f32), _ptr_array(idxs, "idx", torch.int32) if idxs else None,
        _ptr(ws, torch.uint8, name="ws"), ws.numel(), _stream(stream))
    _check(rc, "lstm_bwd_stack")
    return {"dX": dXs, "dW": dWs, "db": dbs, "idx": idxs}


def time_reverse(src, dst=None, stream=None):
    """dst[s] = src[T-1-s] along the first dimension (a new tensor unless given)."""
    if dst is None:
        dst = torch.empty_like(src)
    T = src.shape[0]
    step = src[0].numel() * src.element_size()
    rc = load().lstmss_time_reverse(int(T), int(step), _ptr(src, name="src"),
                                    _ptr(dst, src.dtype, tuple(src.shape), "dst"), _stream(stream))
    _check(rc, "lstmss_time_reverse")
    return dst


def bidir_join(h_fwd, h_rev, out=None, stream=None):
    """[T][2H][B] output of a bidirectional layer: out[t] = [h_fwd[t]; h_rev[T-1-t]]."""
    T, H, B = h_fwd.shape
    d = dims(T, B, 1, H, h_fwd.dtype)
    if out is None:
        out = torch.empty((T, 2 * H, B), dtype=h_fwd.dtype, device=h_fwd.device)
    rc = load().lstmss_bidir_join(ctypes.byref(d), _ptr(h_fwd, name="h_fwd"),
                                  _ptr(h_rev, h_fwd.dtype, (T, H, B), "h_rev"),
                                  _ptr(out, h_fwd.dtype, (T, 2 * H, B), "out"), _stream(stream))
    _check(rc, "lstmss_bidir_join")
    return out


def bwd_bidir(x, x_rev, W_fwd, W_rev, cache_fwd, cache_rev, dH_up, sparsity=0.5, P=4, R=8,
              kind=COARSE, My=0, Mx=0, want_dX=True, out=None, ws=None, stream=None):
    """Backward of a bidirectional layer (both directions concurrently).
    dH_up [T][2H][B].  Returns dict(dX, dW_fwd, dW_rev, db_fwd, db_rev, idx_fwd, idx_rev)."""
    T, I, B = x.shape
    H = W_fwd.shape[0] // 4
    st = x.dtype
    dev = x.device
    f32 = torch.float32
    d = dims(T, B, I, H, st)
    s = structure(P, R, kind, My, Mx) if sparsity > 0 else None
    o = dict(out or {})
    for k, shape, dt in (("dW_fwd", (4 * H, I + H), f32), ("dW_rev", (4 * H, I + H), f32),
                         ("db_fwd", (4 * H,), f32), ("db_rev", (4 * H,), f32)):
        if o.get(k) is None:
            o[k] = torch.empty(shape, dtype=dt, device=dev)
    if want_dX and o.get("dX") is None:
        o["dX"] = torch.empty((T, I, B), dtype=f32, device=dev)
    if s is not None:
        ne = index_entries(d, sparsity, s)
        for k in ("idx_fwd", "idx_rev"):
            if o.get(k) is None:
                o[k] = torch.empty((T, ne), dtype=torch.int32, device=dev)
    if ws is None:
        n = load().lstmss_bidir_workspace_bytes(ctypes.byref(d), float(sparsity),
                                                ctypes.byref(s) if s is not None else None)
        _check(0 if n >= 0 else int(n), "lstmss_bidir_workspace_bytes")
        ws = torch.empty(int(n), dtype=torch.uint8, device=dev)
    rc = load().lstm_bwd_bidir(
        ctypes.byref(d), float(sparsity), ctypes.byref(s) if s is not None else None,
        _ptr(x, st, name="x"), _ptr(x_rev, st, (T, I, B), "x_rev"),
        _ptr(W_fwd, st, (4 * H, I + H), "W_fwd"), _ptr(W_rev, st, (4 * H, I + H), "W_rev"),
        _ptr(cache_fwd, torch.uint8, name="cache_fwd"), _ptr(cache_rev, torch.uint8, name="cache_rev"),
        _ptr(dH_up, f32, (T, 2 * H, B), "dH_up"), _ptr(o.get("dX"), f32, (T, I, B), "dX"),
        _ptr(o["dW_fwd"], f32, name="dW_fwd"), _ptr(o["dW_rev"], f32, name="dW_rev"),
        _ptr(o["db_fwd"], f32, name="db_fwd"), _ptr(o["db_rev"], f32, name="db_rev"),
        _ptr(o.get("idx_fwd"), torch.int32, name="idx_fwd"),
        _ptr(o.get("idx_rev"), torch.int32, name="idx_rev"),
        _ptr(ws, torch.uint8, name="ws"), ws.numel(), _stream(stream))
    _check(rc, "lstm_bwd_bidir")
    return o


def _bwd_outputs(T, B, I, H, dev, want_dX, out):
    out = dict(out or {})
    f32 = torch.float32
    if want_dX and out.get("dX") is None:
        out["dX"] = torch.empty((T, I, B), dtype=f32, device=dev)
    for k, shape in (("dW", (4 * H, I + H)), ("db", (4 * H,)), ("dh0", (H, B)), ("dc0", (H, B))):
        if out.get(k) is None:
            out[k] = torch.empty(shape, dtype=f32, device=dev)
    return out


def bwd_dense(x, W, cache, dH_up, dhT=None, dcT=None, want_dX=True, out=None, ws=None,
              stream=None):
    """Dense backward of one layer.  Returns dict(dX, dW, db, dh0, dc0)."""
    T, I, B = x.shape
    H = W.shape[0] // 4
    st = x.dtype
    d = dims(T, B, I, H, st)
    o = _bwd_outputs(T, B, I, H, x.device, want_dX, out)
    if ws is None:
        ws = torch.empty(workspace_bytes(d, 0.0, None), dtype=torch.uint8, device=x.device)
    f32 = torch.float32
    rc = load().lstm_bwd_dense(
        ctypes.byref(d), _ptr(x, st, name="x"), _ptr(W, st, (4 * H, I + H), "W"),
        _ptr(cache, torch.uint8, name="cache"), _ptr(dH_up, f32, (T, H, B), "dH_up"),
        _ptr(dhT, f32, (H, B), "dhT"), _ptr(dcT, f32, (H, B), "dcT"),
        _ptr(o.get("dX"), f32, (T, I, B), "dX"), _ptr(o["dW"], f32, name="dW"),
        _ptr(o["db"], f32, name="db"), _ptr(o["dh0"], f32, name="dh0"),
        _ptr(o["dc0"], f32, name="dc0"), _ptr(ws, torch.uint8, name="ws"), ws.numel(),
        _stream(stream))
    _check(rc, "lstm_bwd_dense")
    return o


def bwd_structsparse(x, W, cache, dH_up, sparsity=0.5, P=4, R=8, dhT=None, dcT=None,
                     want_dX=True, want_idx=True, want_dbg=False, out=None, ws=None, stream=None,
                     kind=COARSE, My=0, Mx=0):
    """Structurally sparsified backward of one layer (COARSE: P, R; FINE: My, Mx).

    Returns dict(dX, dW, db, dh0, dc0, idx [T][index entries] int32,
    dbg [T][4H][B] or None)."""
    T, I, B = x.shape
    H = W.shape[0] // 4
    st = x.dtype
    d = dims(T, B, I, H, st)
    s = structure(P, R, kind, My, Mx)
    o = _bwd_outputs(T, B, I, H, x.device, want_dX, out)
    ne = index_entries(d, sparsity, s)
    if want_idx and o.get("idx") is None:
        o["idx"] = torch.empty((T, ne), dtype=torch.int32, device=x.device)
    if want_dbg and o.get("dbg") is None:
        o["dbg"] = torch.empty((T, 4 * H, B), dtype=st, device=x.device)
    if ws is None:
        ws = torch.empty(workspace_bytes(d, sparsity, s), dtype=torch.uint8, device=x.device)
    f32 = torch.float32
    rc = load().lstm_bwd_structsparse(
        ctypes.byref(d), float(sparsity), ctypes.byref(s), _ptr(x, st, name="x"),
        _ptr(W, st, (4 * H, I + H), "W"), _ptr(cache, torch.uint8, name="cache"),
        _ptr(dH_up, f32, (T, H, B), "dH_up"), _ptr(dhT, f32, (H, B), "dhT"),
        _ptr(dcT, f32, (H, B), "dcT"), _ptr(o.get("dX"), f32, (T, I, B), "dX"),
        _ptr(o["dW"], f32, name="dW"), _ptr(o["db"], f32, name="db"),
        _ptr(o["dh0"], f32, name="dh0"), _ptr(o["dc0"], f32, name="dc0"),
        _ptr(o.get("idx"), torch.int32, (T, ne), "idx"),
        _ptr(o.get("dbg"), st, (T, 4 * H, B), "dbg"), _ptr(ws, torch.uint8, name="ws"),
        ws.numel(), _stream(stream))
    _check(rc, "lstm_bwd_structsparse")
    return o


def select_compact(dG, sparsity=0.5, P=4, R=8, want_scores=True, stream=None, kind=COARSE,
                   My=0, Mx=0):
    """Score / select / compact one gate-gradient matrix dG [4H][B] with the
    kernels the backward pass runs at this shape (the two-kernel path, with
    its chunk-sum scratch allocated here, at H*B >= 65536).

    COARSE: (kept rows [K'][B], kept slice indices, slice scores [4H/P]).
    FINE: (masked matrix [4H][B], kept block indices [4H/Mx][nb-K],
    block scores [4H/Mx][nb])."""
    G, B = dG.shape
    H = G // 4
    st = dG.dtype
    d = dims(1, B, 1, H, st)
    s = structure(P, R, kind, My, Mx)
    kp = kept_rows(d, sparsity, s)
    ne = index_entries(d, sparsity, s)
    dGc = torch.empty((kp, B), dtype=st, device=dG.device)
    if kind == FINE:
        nb = -(-B // My)
        idx = torch.empty((G // Mx, ne // (G // Mx)), dtype=torch.int32, device=dG.device)
        sc = (torch.empty((G // Mx, nb), dtype=torch.float64, device=dG.device)
              if want_scores else None)
    else:
        idx = torch.empty((ne,), dtype=torch.int32, device=dG.device)
        sc = (torch.empty((G // P,), dtype=torch.float64, device=dG.device)
              if want_scores else None)
    n = select_workspace_bytes(d, sparsity, s)
    ws = torch.empty(n, dtype=torch.uint8, device=dG.device) if n > 0 else None
    rc = load().lstmss_select_compact(ctypes.byref(d), float(sparsity), ctypes.byref(s),
                                      _ptr(dG, st, name="dG"), _ptr(dGc), _ptr(idx), _ptr(sc),
                                      _ptr(ws, torch.uint8, name="ws"),
                                      0 if ws is None else ws.numel(), _stream(stream))
    _check(rc, "lstmss_select_compact")
    return dGc, idx, sc


NOALLOC_SCRATCH_BYTES = 1 << 20


def select_compact_noalloc(dG, dG_c, idx, scores=None, sparsity=0.5, P=4, R=8, stream=None,
                           kind=COARSE, My=0, Mx=0):
    """lstmss_select_compact_noalloc on caller-given outputs (nothing is
    allocated here or in the library): dG [4H][B], dG_c [K'][B] (or the
    masked [4H][B] for FINE), idx, scores (or None)."""
    G, B = dG.shape
    d = dims(1, B, 1, G // 4, dG.dtype)
    s = structure(P, R, kind, My, Mx)
    rc = load().lstmss_select_compact_noalloc(
        ctypes.byref(d), float(sparsity), ctypes.byref(s), _ptr(dG, name="dG"),
        _ptr(dG_c, dG.dtype, name="dG_c"), _ptr(idx, torch.int32, name="idx"),
        _ptr(scores, torch.float64, name="scores"), _stream(stream))
    _check(rc, "lstmss_select_compact_noalloc")


def cache_views(cache, T, B, H, dtype):
    """Views of a cache buffer: gates [T][4H][B], c [T+1][H][B] (fp32), h [T+1][H][B].

    The layout (256-byte aligned sections in this order) is the one
    lstmss_cache_bytes sizes."""
    st = torch_dtype(dtype)
    es = 2 if st == torch.bfloat16 else 4

    def a256(n):
        return (n + 255) // 256 * 256
    g_bytes = T * 4 * H * B * es
    c_off = a256(g_bytes)
    c_bytes = (T + 1) * H * B * 4
    h_off = c_off + a256(c_bytes)
    gates = cache[:g_bytes].view(st).view(T, 4 * H, B)
    c = cache[c_off:c_off + c_bytes].view(torch.float32).view(T + 1, H, B)
    h = cache[h_off:h_off + (T + 1) * H * B * es].view(st).view(T + 1, H, B)
    return gates, c, h


OPTIONS = {"graphs": 0, "side_stream": 1, "stack_dx_steps": 2, "fine_skip": 3, "gemm_dma": 4, "gemm_select": 5,
           "fine_fused": 6, "wgrad_big": 7}


def set_option(name: str, value: int):
    """Execution options of include/lstmss.h (graphs); results are identical
    under every setting."""
    _check(load().lstmss_set_option(OPTIONS[name], int(value)), "lstmss_set_option")


def graphs_enable(on: bool = True):
    set_option("graphs", 1 if on else 0)


def timing_enable(on: bool = True):
    _check(load().lstmss_timing_enable(1 if on else 0), "lstmss_timing_enable")


def timing_reset():
    _check(load().lstmss_timing_reset(), "lstmss_timing_reset")


def timing_read():
    """{kernel kind: (total ms, launches)} accumulated since the last reset."""
    out = {}
    for name, k in KERNEL_KINDS.items():
        ms, n = ctypes.c_double(0), ctypes.c_int64(0)
        _check(load().lstmss_timing_read(k, ctypes.byref(ms), ctypes.byref(n)),
               "lstmss_timing_read")
        out[name] = (ms.value, n.value)
    return out
