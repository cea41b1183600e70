"""Seeded synthetic workloads for the fragment-based image scan.

This module only describes nets (layer lists) and draws their random weights and
images.  It holds none of the scan's arithmetic, so the GPU path and the CPU
oracle can both take their inputs from here without sharing any computation.

Net description: a list of layer dicts
  {"kind": "conv" | "pool" | "fc", "k": int, "c_in": int, "c_out": int,
   "act": "none" | "tanh" | "softmax"}
Convolution weights are OIHW ``[c_out][c_in][k][k]`` float32 (cross-correlation,
no kernel flip), biases ``[c_out]`` float32; pools carry no parameters.  A fully
connected layer is written with the kernel size it has when applied to the map
it receives (the first FC sees a k x k map, later ones a 1 x 1 map), which is
how the paper's Table 1 net and the five workloads below state them.

Random draws follow numpy's PCG64 ``default_rng``: weights with seed = workload
id, then for each parametrised layer in order its weight tensor and then its
bias; the image with seed = 100 + workload id, uniform [0, 1) float32 in
``[B][H][W][C]`` order.  "N(0, s)" means standard deviation s.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np


def _layer(kind, k, c_in, c_out, act, kx):
    L = {"kind": kind, "k": k, "c_in": c_in, "c_out": c_out, "act": act}
    if kx is not None and kx != k:
        L["kx"] = kx  # columns of a rectangular kernel / pool (k: its rows)
    return L


def conv(k, c_in, c_out, act="tanh", kx=None):
    return _layer("conv", k, c_in, c_out, act, kx)


def pool(k, c, kx=None, stride=None, stride_x=None):
    """A k x kx max-pool; stride / stride_x (default: the pool's size, the
    non-overlapping pools of the paper) give the step between windows."""
    L = _layer("pool", k, c, c, "none", kx)
    if stride is not None or stride_x is not None:
        kx_ = L.get("kx", k)
        sy = stride if stride is not None else k
        sx = stride_x if stride_x is not None else (sy if kx_ == k and stride is not None else kx_)
        L["stride"], L["stride_x"] = sy, sx
    return L


def fc(k, c_in, c_out, act="tanh", kx=None):
    return _layer("fc", k, c_in, c_out, act, kx)


def n4_layers():
    """Net N4 of the paper's Table 1 (95x95 greyscale patch, 11 layers)."""
    return [
        conv(4, 1, 48), pool(2, 48),
        conv(5, 48, 48), pool(2, 48),
        conv(4, 48, 48), pool(2, 48),
        conv(4, 48, 48), pool(2, 48),
        fc(3, 48, 200), fc(1, 200, 2, "softmax"),
    ]


@dataclass
class Workload:
    wid: int
    name: str
    layers: list
    patch: int           # w_0 as stated for the workload
    batch: int
    height: int
    width: int
    channels: int
    sigma: float
    zero_bias: bool
    dtype: str           # "f32" or "bf16" (storage / MFMA operand type)
    note: str = ""
    extra: dict = field(default_factory=dict)

    @property
    def out_h(self):
        return self.height - self.patch + 1

    @property
    def out_w(self):
        return self.width - self.patch + 1

    @property
    def n_classes(self):
        return self.layers[-1]["c_out"]


WORKLOADS = {
    1: Workload(1, "tiny_64", [
        conv(3, 1, 4), pool(2, 4), conv(3, 4, 8), pool(2, 8),
        fc(2, 8, 16), fc(1, 16, 2, "softmax")],
        patch=14, batch=1, height=64, width=64, channels=1,
        sigma=0.1, zero_bias=True, dtype="f32",
        note="tiny net, 14x14 patch, 1x64x64x1 image"),
    2: Workload(2, "n4_512", n4_layers(), patch=95, batch=1, height=512,
                width=512, channels=1, sigma=0.05, zero_bias=False, dtype="f32",
                note="net N4 (Table 1), 95x95 patch, 1x512x512x1 image"),
    3: Workload(3, "rgb5pool_2048", [
        conv(2, 3, 16), pool(2, 16), conv(3, 16, 16), pool(2, 16),
        conv(3, 16, 16), pool(2, 16), conv(2, 16, 16), pool(2, 16),
        conv(2, 16, 16), pool(2, 16),
        fc(2, 16, 100), fc(1, 100, 2, "softmax")],
        patch=101, batch=1, height=2048, width=2048, channels=3,
        sigma=0.05, zero_bias=False, dtype="f32",
        note="5-pool RGB net, 101x101 patch, 1x2048x2048x3 image"),
    4: Workload(4, "n4_8x1024", n4_layers(), patch=95, batch=8, height=1024,
                width=1024, channels=1, sigma=0.05, zero_bias=False, dtype="f32",
                note="net N4, batch of 8 1024x1024 greyscale images"),
    5: Workload(5, "mixed_bf16_1536", [
        conv(3, 3, 32, "none"), conv(3, 32, 32), pool(3, 32),
        conv(4, 32, 64), pool(2, 64), conv(3, 64, 64), pool(2, 64),
        fc(3, 64, 128), fc(1, 128, 4, "softmax")],
        patch=61, batch=1, height=1536, width=1536, channels=3,
        sigma=0.05, zero_bias=False, dtype="bf16",
        note="mixed-order net in bf16 (fp32 accumulate), 1x1536x1536x3 image; "
             "the layer stack fixes the patch at 61 (the stated 57 does not "
             "divide at the 3x3 pool)",
        extra={"stated_patch": 57}),
}


def make_weights(layers, seed, sigma, zero_bias=False):
    """Return a list with, per layer, (weight OIHW f32, bias f32) or None."""
    rng = np.random.default_rng(seed)
    params = []
    for L in layers:
        if L["kind"] == "pool":
            params.append(None)
            continue
        ky, kx, ci, co = L["k"], L.get("kx", L["k"]), L["c_in"], L["c_out"]
        w = rng.normal(0.0, sigma, size=(co, ci, ky, kx)).astype(np.float32)
        if zero_bias:
            b = np.zeros(co, np.float32)
        else:
            b = rng.normal(0.0, sigma, size=(co,)).astype(np.float32)
        params.append((w, b))
    return params


def make_image(seed, batch, height, width, channels):
    rng = np.random.default_rng(seed)
    return rng.random((batch, height, width, channels), dtype=np.float32)


def workload_inputs(wid, batch=None, height=None, width=None):
    """Weights and image of workload ``wid``; the image size may be overridden
    (parity tests scan smaller images with the same net and weights)."""
    w = WORKLOADS[wid]
    params = make_weights(w.layers, seed=wid, sigma=w.sigma, zero_bias=w.zero_bias)
    img = make_image(100 + wid, batch or w.batch, height or w.height,
                     width or w.width, w.channels)
    return params, img


def random_net(rng, max_layers=6, max_c=6, allow_pools=True):
    """A random conv/pool/fc stack for property tests.  Kernel and pool sizes are
    drawn so that every pool divides its map; the patch size is built bottom-up
    from a final 1x1 map, and returned with the layers."""
    # Build the stack top-down in patch-map sizes: start from the FC head.
    n_cls = int(rng.integers(2, 4))
    c = int(rng.integers(1, max_c + 1))
    c_in0 = c
    layers = []
    n_body = int(rng.integers(1, max_layers))
    for _ in range(n_body):
        if allow_pools and rng.random() < 0.45:
            layers.append(pool(int(rng.integers(2, 4)), c))
        else:
            co = int(rng.integers(1, max_c + 1))
            layers.append(conv(int(rng.integers(1, 4)), c, co,
                               "tanh" if rng.random() < 0.7 else "none"))
            c = co
    hidden = int(rng.integers(2, 7))
    layers.append({"kind": "fc", "k": 0, "c_in": c, "c_out": hidden, "act": "tanh"})
    layers.append(fc(1, hidden, n_cls, "softmax"))
    # Size the patch from the top: the map entering the first FC is w_L; any
    # w_L works as long as every pool divides its input, so grow downward.
    w_L = int(rng.integers(1, 4))
    w = w_L
    for L in reversed(layers[:-2]):
        if L["kind"] == "pool":
            w = w * L["k"]
        else:
            w = w + L["k"] - 1
    layers[-2]["k"] = w_L
    return layers, w, c_in0


def random_rect_net(rng, max_layers=6, max_c=5):
    """A random stack with rectangular kernels and pools (k: rows, kx:
    columns, drawn independently).  Returns (layers, (h0, w0), c_in)."""
    n_cls = int(rng.integers(2, 4))
    c = int(rng.integers(1, max_c + 1))
    c_in0 = c
    layers = []
    for _ in range(int(rng.integers(1, max_layers))):
        if rng.random() < 0.45:
            ky, kx = int(rng.integers(1, 4)), int(rng.integers(1, 4))
            if ky * kx == 1:
                kx = 2
            layers.append(pool(ky, c, kx=kx))
        else:
            co = int(rng.integers(1, max_c + 1))
            layers.append(conv(int(rng.integers(1, 5)), c, co, "tanh" if rng.random() < 0.7 else "none",
                               kx=int(rng.integers(1, 5))))
            c = co
    hidden = int(rng.integers(2, 6))
    hy, hx = int(rng.integers(1, 4)), int(rng.integers(1, 4))
    layers.append(fc(hy, c, hidden, "tanh", kx=hx))
    layers.append(fc(1, hidden, n_cls, "softmax"))
    h, w = hy, hx
    for L in reversed(layers[:-2]):
        ky, kx = L["k"], L.get("kx", L["k"])
        if L["kind"] == "pool":
            h, w = h * ky, w * kx
        else:
            h, w = h + ky - 1, w + kx - 1
    return layers, (h, w), c_in0


def random_stride_net(rng, max_layers=6, max_c=5):
    """A random stack whose pools may overlap (stride below the size) or
    leave gaps (stride above it), square or rectangular.  Returns (layers,
    (h0, w0), c_in)."""
    n_cls = int(rng.integers(2, 4))
    c = int(rng.integers(1, max_c + 1))
    c_in0 = c
    layers = []
    for _ in range(int(rng.integers(1, max_layers))):
        if rng.random() < 0.5:
            ky, kx = int(rng.integers(1, 5)), int(rng.integers(1, 5))
            sy, sx = int(rng.integers(1, 4)), int(rng.integers(1, 4))
            layers.append(pool(ky, c, kx=kx, stride=sy, stride_x=sx))
        else:
            co = int(rng.integers(1, max_c + 1))
            layers.append(conv(int(rng.integers(1, 4)), c, co, "tanh" if rng.random() < 0.7 else "none",
                               kx=int(rng.integers(1, 4))))
            c = co
    hidden = int(rng.integers(2, 6))
    hy, hx = int(rng.integers(1, 4)), int(rng.integers(1, 4))
    layers.append(fc(hy, c, hidden, "tanh", kx=hx))
    layers.append(fc(1, hidden, n_cls, "softmax"))
    h, w = hy, hx
    for L in reversed(layers[:-2]):
        ky, kx = L["k"], L.get("kx", L["k"])
        if L["kind"] == "pool":
            h, w = (h - 1) * L.get("stride", ky) + ky, (w - 1) * L.get("stride_x", kx) + kx
        else:
            h, w = h + ky - 1, w + kx - 1
    return layers, (h, w), c_in0
