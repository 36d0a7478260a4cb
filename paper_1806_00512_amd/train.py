"""Dense-after-sparse training of an LSTM layer stack on the GPU.

The method's training procedure (section 5, Table 2): the first steps run the
structurally sparsified backward pass, the rest the dense one, with the total
number of steps unchanged; the paper reports a 3-to-1 ratio of sparse to
dense steps as enough to recover the dense model's quality.

One training step here:
  forward of every layer (bottom first) into its backward cache,
  loss gradient at the top (synthetic regression target; see
  lstmss_mse_grad),
  backward of every layer as one wavefront stack call (lstm_bwd_stack: a
  layer's input gradient is the upstream gradient of the layer below, the
  layers overlap in time; the bottom layer's input gradient is not formed),
  SGD update of every layer's W and b.

Every step runs in liblstmss kernels through the C ABI; this module holds the
buffers and the schedule.  All buffers are allocated once.
"""
from __future__ import annotations

from dataclasses import dataclass

import torch

from . import lstmss as L


def dense_after_sparse(total_steps: int, sparse_fraction: float = 0.75) -> list:
    """Schedule of `total_steps` steps: the first round(sparse_fraction * total)
    sparse (True), the rest dense (False)."""
    if total_steps < 0 or not 0.0 <= sparse_fraction <= 1.0:
        raise ValueError("need total_steps >= 0 and 0 <= sparse_fraction <= 1")
    n_sparse = int(round(sparse_fraction * total_steps))
    return [True] * n_sparse + [False] * (total_steps - n_sparse)


@dataclass
class StackConfig:
    layers: int
    input_size: int
    hidden: int
    batch: int
    steps: int                     # sequence length T
    dtype: torch.dtype = torch.float32
    lr: float = 0.1
    sparsity: float = 0.5
    P: int = 4                     # coarse structure (kind COARSE)
    R: int = 8
    kind: int = L.COARSE
    My: int = 0                    # fine structure (kind FINE)
    Mx: int = 0

    def layer_input(self, l: int) -> int:
        return self.input_size if l == 0 else self.hidden

    def structure_kw(self) -> dict:
        if self.kind == L.FINE:
            return {"kind": L.FINE, "My": self.My, "Mx": self.Mx}
        return {"P": self.P, "R": self.R}


class StackTrainer:
    """Trains Ws[l] ([4H][I_l+H], storage dtype) and bs[l] ([4H] fp32) in place."""

    def __init__(self, cfg: StackConfig, Ws, bs, device="cuda:0"):
        L.load()
        self.cfg = cfg
        self.Ws, self.bs = list(Ws), list(bs)
        dev = torch.device(device)
        T, B, H = cfg.steps, cfg.batch, cfg.hidden
        f32 = torch.float32
        self.caches, self.fws, self.houts = [], [], []
        self.outs, self.idx, ds = [], [], []
        skw = cfg.structure_kw()
        self.structure = L.structure(**skw)
        for l in range(cfg.layers):
            I = cfg.layer_input(l)
            d = L.dims(T, B, I, H, cfg.dtype)
            if tuple(self.Ws[l].shape) != (4 * H, I + H) or self.Ws[l].dtype != cfg.dtype:
                raise ValueError("W[%d] must be [%d][%d] %s" % (l, 4 * H, I + H, cfg.dtype))
            self.caches.append(torch.empty(L.cache_bytes(d), dtype=torch.uint8, device=dev))
            self.fws.append(torch.empty(L.fwd_workspace_bytes(d), dtype=torch.uint8, device=dev))
            self.houts.append(torch.empty((T, H, B), dtype=cfg.dtype, device=dev))
            ds.append(d)
            o = {"dW": torch.empty((4 * H, I + H), dtype=f32, device=dev),
                 "db": torch.empty(4 * H, dtype=f32, device=dev)}
            if l > 0:
                o["dX"] = torch.empty((T, I, B), dtype=f32, device=dev)
            self.outs.append(o)
            self.idx.append(torch.empty((T, L.index_entries(d, cfg.sparsity, self.structure)),
                                        dtype=torch.int32, device=dev))
        self.sp_ws = torch.empty(L.stack_workspace_bytes(ds, cfg.sparsity, self.structure),
                                 dtype=torch.uint8, device=dev)
        self.dn_ws = torch.empty(L.stack_workspace_bytes(ds, 0.0, None), dtype=torch.uint8,
                                 device=dev)
        self.dH = torch.empty((T, H, B), dtype=f32, device=dev)
        self.loss = torch.empty(L.LOSS_SLOTS, dtype=torch.float64, device=dev)

    def forward(self, x):
        inp = x
        for l in range(self.cfg.layers):
            L.fwd_cache(inp, self.Ws[l], self.bs[l], h_out=self.houts[l], cache=self.caches[l],
                        ws=self.fws[l])
            inp = self.houts[l]
        return inp

    def step(self, x, y, sparse: bool):
        """One training step; returns the device fp64 loss slot (before the update)."""
        cfg = self.cfg
        top = self.forward(x)
        L.mse_grad(top, y, dH=self.dH, loss=self.loss)
        xs = [x] + self.houts[:-1]
        L.bwd_stack(xs, self.Ws, self.caches, self.dH,
                    sparsity=cfg.sparsity if sparse else 0.0,
                    dXs=[o.get("dX") for o in self.outs], dWs=[o["dW"] for o in self.outs],
                    dbs=[o["db"] for o in self.outs], idxs=self.idx if sparse else None,
                    ws=self.sp_ws if sparse else self.dn_ws, **cfg.structure_kw())
        for l in range(cfg.layers):
            L.sgd_update(self.Ws[l], self.bs[l], self.outs[l]["dW"], self.outs[l]["db"], cfg.lr,
                         cfg.layer_input(l))
        return self.loss[-1:]

    def train(self, x, y, schedule):
        """Run the schedule (list of bools, True = sparse step); returns the
        per-step losses as a device tensor."""
        losses = torch.empty(len(schedule), dtype=torch.float64, device=self.loss.device)
        for i, sparse in enumerate(schedule):
            losses[i:i + 1].copy_(self.step(x, y, sparse))
        return losses
