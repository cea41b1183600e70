"""Pins for the mirrored-border oracle (Section 3.2: the image's edges are
mirrored so that the net applies at every position).  CPU only."""
import json
import os

import numpy as np
import pytest

import oracle
from oracle import border as ob
from paper_1302_1700_amd import workloads as wl

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "mirror_border.json")


def _golden():
    with open(GOLDEN) as f:
        return json.load(f)


@pytest.mark.parametrize("mode", ["reflect", "symmetric"])
def test_mirror_index_sequences(mode):
    """The extension reads the hand-derived image indices, including a border
    wider than the image (repeated mirroring) and a one-pixel image."""
    for case in _golden()["cases"]:
        n, lo, hi = case["n"], case["before"], case["after"]
        img = np.arange(n, dtype=np.float64).reshape(1, n, 1, 1)
        # a w_0 whose widths are (lo, hi) exists only for hi in {lo, lo + 1};
        # check the index map itself through the padding primitive
        got = np.pad(img, ((0, 0), (lo, hi), (0, 0), (0, 0)), mode=mode)[0, :, 0, 0]
        assert got.astype(int).tolist() == case[mode], (case, mode)
        if hi in (lo, lo + 1):
            w0 = lo + hi + 1
            assert ob.border_widths(w0) == (lo, hi)
            ext = ob.mirror_pad(np.broadcast_to(img, (1, n, n, 1)), w0, mode)
            assert ext[0, :, 0, 0].astype(int).tolist() == case[mode]


def test_border_widths():
    for w0, (lo, hi) in _golden()["widths"].items():
        assert ob.border_widths(int(w0)) == (lo, hi)


def _interior_check(layers, params, img, w0, mode, widths=None):
    """Mirrored output (y, x) = the valid scan's output (y - p0, x - p0) for
    every window that lies inside the image."""
    full = ob.scan_mirrored(layers, params, img, w0, mode)
    valid = oracle.patch_forward(layers, params, img, w0)
    p0 = (widths or ob.border_widths(w0))[0]
    B, H, W, _ = img.shape
    assert full.shape == (B, H, W, valid.shape[-1])
    inner = full[:, p0:p0 + H - w0 + 1, p0:p0 + W - w0 + 1]
    return np.abs(inner - valid).max()


@pytest.mark.parametrize("mode", ["reflect", "symmetric"])
def test_interior_equals_valid_scan_even_patch(mode):
    w = wl.WORKLOADS[1]  # w_0 = 14: p0 = 6 before, 7 after
    params, img = wl.workload_inputs(1, height=25, width=22)
    assert _interior_check(w.layers, params, img, w.patch, mode) <= 1e-12


def test_interior_equals_valid_scan_odd_patch():
    layers = [wl.conv(2, 2, 3), wl.pool(2, 3), wl.fc(2, 3, 4), wl.fc(1, 4, 2, "softmax")]
    params = wl.make_weights(layers, 31, 0.5)
    img = wl.make_image(32, 2, 13, 11, 2)
    w0 = 5
    assert _interior_check(layers, params, img, w0, "reflect") <= 1e-12


def test_planted_mistakes_are_caught():
    """Swapping the before / after widths of an even patch, or the mirror
    type, changes the results the pins fix."""
    w = wl.WORKLOADS[1]
    params, img = wl.workload_inputs(1, height=25, width=22)
    lo, hi = ob.border_widths(w.patch)
    assert _interior_check(w.layers, params, img, w.patch, "reflect", widths=(hi, lo)) > 1e-3
    a = ob.scan_mirrored(w.layers, params, img, w.patch, "reflect")
    b = ob.scan_mirrored(w.layers, params, img, w.patch, "symmetric")
    assert np.abs(a - b).max() > 1e-3
    # the reflect sequence is not the symmetric one
    case = _golden()["cases"][0]
    assert case["reflect"] != case["symmetric"]
