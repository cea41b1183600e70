"""Pins for the oracle's algorithmic work count (oracle.index.algorithmic_flops).

The count is the numerator of every TFLOP/s figure, so it is pinned to facts
that do not come from its own recursion:

  - a closed form per axis.  Summed over the fragments, a k-wide layer (a
    convolution, Eqs. 3-4, or a pool, Eqs. 6-7: sum over o < k of
    div(s - o, k) = s - (k - 1); for a pool of stride t, sum over o < t of
    div(s - o - k + t, t) = s - (k - 1) likewise) removes k - 1 pixels from
    every fragment,
    so the total width after layer l is W - sum_{m <= l} (k_m - 1) * Q_m,
    with Q_m the fragments per axis entering layer m (the size of the map of
    the same layer applied with dilation Q_m, and the final total is the
    number of windows, W - w_0 + 1: the fragments cover every window exactly
    once, Section 3).  Sizes are separable, so the pixels of a layer are the
    product of its two axis totals;
  - hand counts (tests/golden/flops_hand.json);
  - planted mistakes in a copy of the oracle's source (input-side instead of
    output-side sizes, a dropped kernel axis, a dropped batch factor), each of
    which must fail one of the pins above.
"""
import importlib.util
import json
import os

import numpy as np
import pytest

from oracle import index as ix
from paper_1302_1700_amd import workloads as wl

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(os.path.dirname(HERE), "oracle", "index.py")


def closed_form(layers, B, H, W):
    """Per layer, B * T_y * T_x * 2 * c_in * k_y * k_x * c_out with the
    per-axis totals T of the docstring, and the final totals (T_y, T_x).
    Valid when no fragment runs empty (H - h_0 + 1 >= S_y and likewise for
    the columns)."""
    Qy = Qx = 1
    Ty, Tx = H, W
    res = []
    for L in layers:
        ky, kx = L["k"], L.get("kx", L["k"])
        Ty -= (ky - 1) * Qy
        Tx -= (kx - 1) * Qx
        if L["kind"] == "pool":  # its stride, the fragments' step (its size unless given)
            Qy, Qx = Qy * L.get("stride", ky), Qx * L.get("stride_x", kx)
            res.append(0)
        else:
            res.append(B * Ty * Tx * 2 * L["c_in"] * ky * kx * L["c_out"])
    return res, (Ty, Tx)


def _strides(layers):
    Sy = Sx = 1
    for L in layers:
        if L["kind"] == "pool":
            Sy, Sx = Sy * ix.syx(L)[0], Sx * ix.syx(L)[1]
    return Sy, Sx


def _cases():
    """(layers, B, H, W): the five workload nets at full size and random
    square and rectangular nets on images where every fragment holds a
    window."""
    out = []
    for w in wl.WORKLOADS.values():
        out.append((w.layers, w.batch, w.height, w.width))
    rng = np.random.default_rng(9100)
    for n in range(45):
        if n % 3 == 2:
            layers, (h0, w0), _ = wl.random_stride_net(rng)
        elif n % 3 == 1:
            layers, (h0, w0), _ = wl.random_rect_net(rng)
        else:
            layers, w0, _ = wl.random_net(rng)
            h0 = w0
        Sy, Sx = _strides(layers)
        B = 1 + n % 3
        out.append((layers, B, h0 + Sy - 1 + int(rng.integers(0, 30)), w0 + Sx - 1 + int(rng.integers(0, 30))))
    return out


def _golden():
    with open(os.path.join(HERE, "golden", "flops_hand.json")) as f:
        g = json.load(f)
    cases = []
    for c in g["cases"]:
        layers = []
        for kind, k, kx, ci, co in c["net"]:
            layers.append({"kind": kind, "k": k, "kx": kx, "c_in": ci, "c_out": co, "act": "none"})
        cases.append((layers, c["batch"], c["height"], c["width"], c["per_layer"], c["total"]))
    return cases


def _pins_fail(mod):
    """True if the module's algorithmic_flops fails any pin."""
    for layers, B, H, W in _cases():
        want, (Ty, Tx) = closed_form(layers, B, H, W)
        h0, w0 = ix.patch_hw(layers)
        if (Ty, Tx) != (H - h0 + 1, W - w0 + 1):
            return True  # (the closed form itself: checked in its own test)
        if list(mod.algorithmic_flops(layers, B, H, W)) != want:
            return True
    for layers, B, H, W, per_layer, total in _golden():
        got = list(mod.algorithmic_flops(layers, B, H, W))
        if got != per_layer or sum(got) != total:
            return True
    return False


def test_closed_form_final_total_is_window_count():
    """The per-axis closed form ends at the number of windows per axis (every
    window is covered exactly once), for every case the pins use."""
    for layers, B, H, W in _cases():
        _, (Ty, Tx) = closed_form(layers, B, H, W)
        h0, w0 = ix.patch_hw(layers)
        assert (Ty, Tx) == (H - h0 + 1, W - w0 + 1)


def test_algorithmic_flops_closed_form():
    for layers, B, H, W in _cases():
        want, _ = closed_form(layers, B, H, W)
        assert list(ix.algorithmic_flops(layers, B, H, W)) == want


def test_fc_layers_count_one_pixel_per_window():
    """Fully connected layers see one pixel per window: B * n_y * n_x *
    2 * c_in * k_y * k_x * c_out (the fragments are a bijection onto the
    windows)."""
    for w in wl.WORKLOADS.values():
        got = ix.algorithmic_flops(w.layers, w.batch, w.height, w.width)
        n = w.batch * w.out_h * w.out_w
        for L, v in zip(w.layers, got):
            if L["kind"] == "fc":
                assert v == n * 2 * L["c_in"] * L["k"] * L.get("kx", L["k"]) * L["c_out"]


def test_algorithmic_flops_hand_counts():
    for layers, B, H, W, per_layer, total in _golden():
        got = list(ix.algorithmic_flops(layers, B, H, W))
        assert got == per_layer and sum(got) == total


def _load_mutant(tmp_path, name, old, new):
    src = open(SRC).read()
    assert src.count(old) == 1, name
    p = tmp_path / ("index_%s.py" % name)
    p.write_text(src.replace(old, new))
    spec = importlib.util.spec_from_file_location("index_" + name, str(p))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


FLOP_MUTATIONS = {
    "input_side_extents": ("pix = sum(sy * sx for (sy, sx) in ext[l + 1])",
                           "pix = sum(sy * sx for (sy, sx) in ext[l])"),
    "kernel_columns_dropped": ('2 * L["c_in"] * kyx(L)[0] * kyx(L)[1] * L["c_out"]',
                               '2 * L["c_in"] * kyx(L)[0] * kyx(L)[0] * L["c_out"]'),
    "batch_dropped": ("res.append(B * pix * 2", "res.append(pix * 2"),
    "multiply_add_as_one": ("res.append(B * pix * 2 *", "res.append(B * pix * 1 *"),
}


def test_unmutated_index_passes(tmp_path):
    mod = _load_mutant(tmp_path, "clean", "import numpy as np", "import numpy as np")
    assert not _pins_fail(mod)


@pytest.mark.parametrize("name", sorted(FLOP_MUTATIONS))
def test_planted_flop_mistake_is_caught(tmp_path, name):
    old, new = FLOP_MUTATIONS[name]
    assert _pins_fail(_load_mutant(tmp_path, name, old, new)), name
