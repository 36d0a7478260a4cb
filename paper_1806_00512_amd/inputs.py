"""Seeded synthetic inputs for the LSTM workloads.

This module holds no arithmetic of the method: it only names the workload
shapes and draws random tensors.  Both the GPU path and the CPU oracle are fed
the identical arrays it returns, so it must not import either of them.

Draw order (numpy ``Generator(PCG64(seed))``, float32): W of every layer
(bottom layer first), then the layer-1 input x, then the upstream gradient of
the top layer's hidden states dH_up.  Biases are zero, h0 = c0 = 0.  For a bf16
workload W and x are rounded to the nearest bfloat16 (ties to even) after the
draw, so they are exactly representable in the storage type.

Layouts: x [T][I][B], W [4H][I+H] (rows i, f, g, o; columns [x | h]),
dH_up [T][H][B]; batch is the contiguous dimension everywhere.

The workloads stand in for the paper's (word language model and NMT LSTMs of
512 cells; section 4): the paper states that the backward-pass speedup depends
only on the layer shape and the sparsity (section 5.5), so random tensors of the
same shapes measure the same thing.
"""
from __future__ import annotations

from dataclasses import dataclass, field, replace

import numpy as np


@dataclass(frozen=True)
class Workload:
    name: str
    layers: int
    input_size: int
    hidden: int
    batch: int
    steps: int
    dtype: str            # "f32" or "bf16" (storage; accumulation is fp32)
    w_scale: float        # W ~ U(-w_scale, w_scale)
    x_std: float          # x ~ N(0, x_std^2)
    up_std: float         # dH_up ~ N(0, up_std^2)
    sparsity: float = 0.5
    sweep: tuple = field(default_factory=tuple)
    P: int = 4
    R: int = 8

    def layer_input(self, layer: int) -> int:
        return self.input_size if layer == 0 else self.hidden

    def truncated(self, steps: int) -> "Workload":
        return replace(self, steps=steps)


WORKLOADS = {
    # 1-layer LSTM, input 128, H 128, batch 16, 20 steps (small case the oracle finishes in seconds)
    "lstm1_h128_b16_t20_f32": Workload("lstm1_h128_b16_t20_f32", 1, 128, 128, 16, 20, "f32",
                                       0.1, 1.0, 1.0),
    # 2-layer word-language-model shape: input = H = 650, batch 20, 35 steps
    "lstm2_lm_h650_b20_t35_f32": Workload("lstm2_lm_h650_b20_t35_f32", 2, 650, 650, 20, 35, "f32",
                                          0.05, 1.0, 0.1),
    # 2-layer LSTM, input = H = 1024, batch 64, 35 steps, sparsity sweep 0/25/50/75 %
    "lstm2_h1024_b64_t35_f32": Workload("lstm2_h1024_b64_t35_f32", 2, 1024, 1024, 64, 35, "f32",
                                        0.05, 1.0, 0.1, sweep=(0.0, 0.25, 0.5, 0.75)),
    # 4-layer seq2seq-encoder shape: input = H = 2048, batch 128, 50 steps
    "lstm4_enc_h2048_b128_t50_f32": Workload("lstm4_enc_h2048_b128_t50_f32", 4, 2048, 2048, 128,
                                             50, "f32", 0.08, 1.0, 0.1),
    # 1-layer input = H = 4096, batch 256, 100 steps, bf16 storage, mixed 9 sparse : 1 dense
    "lstm1_h4096_b256_t100_bf16": Workload("lstm1_h4096_b256_t100_bf16", 1, 4096, 4096, 256, 100,
                                           "bf16", 0.08, 1.0, 0.1),
}
ORDER = list(WORKLOADS)


def round_bf16_f32(a: np.ndarray) -> np.ndarray:
    """Nearest bfloat16 (ties to even) of finite float32 values, kept as float32."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) & 0xFFFF0000
    return u.astype(np.uint32).view(np.float32)


def make_inputs(wl: Workload, seed: int = 0):
    """Return dict(Ws=[...], bs=[...], x=..., dH_up=...) as float32 numpy arrays."""
    rng = np.random.Generator(np.random.PCG64(seed))
    Ws, bs = [], []
    for layer in range(wl.layers):
        I = wl.layer_input(layer)
        shape = (4 * wl.hidden, I + wl.hidden)
        W = rng.random(shape, dtype=np.float32) * np.float32(2 * wl.w_scale) - np.float32(wl.w_scale)
        if wl.dtype == "bf16":
            W = round_bf16_f32(W)
        Ws.append(W)
        bs.append(np.zeros(4 * wl.hidden, dtype=np.float32))
    x = rng.standard_normal((wl.steps, wl.input_size, wl.batch), dtype=np.float32)
    x *= np.float32(wl.x_std)
    if wl.dtype == "bf16":
        x = round_bf16_f32(x)
    dH_up = rng.standard_normal((wl.steps, wl.hidden, wl.batch), dtype=np.float32)
    dH_up *= np.float32(wl.up_std)
    return {"Ws": Ws, "bs": bs, "x": x, "dH_up": dH_up}


def make_target(wl: Workload, seed: int = 1, std: float = 0.5) -> np.ndarray:
    """Synthetic regression target y [T][H][B] for the top layer (float32)."""
    rng = np.random.Generator(np.random.PCG64(seed))
    y = rng.standard_normal((wl.steps, wl.hidden, wl.batch), dtype=np.float32)
    return y * np.float32(std)


def make_layer(T: int, B: int, I: int, H: int, seed: int, w_scale: float = 0.1,
               up_std: float = 1.0, dtype: str = "f32", state: bool = False):
    """One layer of random inputs of any shape (used for edge cases).

    With ``state`` the initial states h0, c0 and the late-time gradients dhT,
    dcT are drawn too (otherwise they are zero / absent)."""
    rng = np.random.Generator(np.random.PCG64(seed))
    W = rng.random((4 * H, I + H), dtype=np.float32) * np.float32(2 * w_scale) - np.float32(w_scale)
    b = (rng.random(4 * H, dtype=np.float32) - np.float32(0.5)) * np.float32(0.2)
    x = rng.standard_normal((T, I, B), dtype=np.float32)
    dH_up = rng.standard_normal((T, H, B), dtype=np.float32) * np.float32(up_std)
    if dtype == "bf16":
        W, x = round_bf16_f32(W), round_bf16_f32(x)
    out = {"W": W, "b": b, "x": x, "dH_up": dH_up, "h0": None, "c0": None, "dhT": None,
           "dcT": None}
    if state:
        h0 = rng.standard_normal((H, B), dtype=np.float32) * np.float32(0.5)
        out["h0"] = round_bf16_f32(h0) if dtype == "bf16" else h0
        out["c0"] = rng.standard_normal((H, B), dtype=np.float32) * np.float32(0.5)
        out["dhT"] = rng.standard_normal((H, B), dtype=np.float32) * np.float32(up_std)
        out["dcT"] = rng.standard_normal((H, B), dtype=np.float32) * np.float32(up_std)
    return out
