"""Pins of the CPU oracle against what the paper and the mathematics fix.

Runs on the CPU.  Each test names the passage it follows.
"""
import json
import math
import os

import numpy as np
import pytest

import oracle
from oracle import index as ix
from paper_1302_1700_amd import workloads as wl

from helpers import dilated_scan, torch_patch_net

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _gold(name):
    with open(os.path.join(GOLD, name)) as f:
        return json.load(f)


# ---- Table 1: patch-level sizes (Sections 2.1.1, 2.1.2) -------------------

def test_table1_patch_sizes():
    g = _gold("table1_n4.json")
    layers = wl.n4_layers()
    sizes = ix.patch_sizes(layers, 95)
    assert sizes == [e["size"] for e in g["layers"]]
    assert ix.patch_size(layers) == 95
    # maps per layer as printed
    maps = [1] + [L["c_out"] for L in layers]
    assert maps == [e["maps"] for e in g["layers"]]
    assert ix.n_fragments(layers) == g["final_fragments"]
    ext = ix.fragment_extents(layers, 512, 512)
    assert len(ext[8]) == 256


def test_workload_output_sizes():
    """Output map sizes (H - w_0 + 1) of the five workloads; workload 5's stack
    fixes its patch at 61 (the stated 57 cannot pass its 3x3 pool)."""
    want = {1: 51, 2: 418, 3: 1948, 4: 930, 5: 1476}
    for wid, w in wl.WORKLOADS.items():
        assert ix.patch_size(w.layers) == w.patch
        assert w.height - w.patch + 1 == want[wid]
        ix.patch_sizes(w.layers, w.patch)
    with pytest.raises(ValueError):
        ix.patch_sizes(wl.WORKLOADS[5].layers, 57)


# ---- Section 2.2.2: offset order; Section 3: fragment count ---------------

def test_offset_order_k2():
    g = _gold("offsets_k2.json")
    layers = [wl.pool(2, 1), wl.fc(1, 1, 1, "none")]
    tab = ix.fragment_table(layers, 9, 9)
    got = [tuple(tab[f]["offsets"][0]) for f in range(4)]
    assert got == [tuple(o) for o in g["offsets"]]
    # base output pixel of child (o_x, o_y) is (o_y, o_x)
    assert [tab[f]["base"] for f in range(4)] == [(0, 0), (0, 1), (1, 0), (1, 1)]


@pytest.mark.parametrize("seed", range(20))
def test_fragment_count_law(seed):
    rng = np.random.default_rng(seed)
    layers, w0, _ = wl.random_net(rng)
    prod = 1
    for L in layers:
        if L["kind"] == "pool":
            prod *= L["k"] ** 2
    H, W = w0 + int(rng.integers(0, 9)), w0 + int(rng.integers(0, 9))
    ext = ix.fragment_extents(layers, H, W)
    assert len(ext[-1]) == prod == ix.n_fragments(layers)


# ---- Sections 3 and 3.1: extents, coverage -------------------------------

@pytest.mark.parametrize("seed", range(30))
def test_extents_spread_and_coverage(seed):
    rng = np.random.default_rng(100 + seed)
    layers, w0, _ = wl.random_net(rng)
    H = w0 + int(rng.integers(0, 13))
    W = w0 + int(rng.integers(0, 13))
    ext = ix.fragment_extents(layers, H, W)
    # sizes of fragments in one layer differ by at most one pixel per axis
    for frags in ext:
        ys = [e[0] for e in frags]
        xs = [e[1] for e in frags]
        assert max(ys) - min(ys) <= 1 and max(xs) - min(xs) <= 1
    # every patch lands on exactly one (fragment, position) of the last layer,
    # and every position inside a final fragment's extent is some patch
    idx = ix.reassembly_index(layers, H, W).reshape(-1, 3)
    keys = set(map(tuple, idx.tolist()))
    assert len(keys) == idx.shape[0] == (H - w0 + 1) * (W - w0 + 1)
    final = ext[-1]
    for (f, y, x) in keys:
        assert y < final[f][0] and x < final[f][1]
    assert sum(a * b for a, b in final) == len(keys)
    tab = ix.fragment_table(layers, H, W)
    for f, e in tab.items():
        assert e["size"] == final[f]


def test_table2_flops():
    g = _gold("table2_flops.json")
    tp = ti = 0.0
    for (l, s, s_prev, pp, pl, w, k, F, fp, fi, sp) in g["rows"]:
        p = ix.flops_patch(s, pp, pl, w, k) / 1e9
        i = ix.flops_image(s_prev, s_prev, pp, pl, F, k) / 1e9
        assert round(p) == fp or math.floor(p) == fp
        assert round(i, 1) == fi
        if l in (3, 5):
            assert round(p / i, 1) == sp
        elif l == 7:
            assert math.floor(p / i * 10) / 10 == sp
        else:  # layer 1: printed 7114.8 does not follow from its columns
            assert round(p / i, 1) == 7100.5
        tp += p
        ti += i
    assert round(tp) == g["total"]["flops_patch_1e9"] + 1 or round(tp) == g["total"]["flops_patch_1e9"]
    assert round(ti, 1) == g["total"]["flops_image_1e9"]
    assert round(tp / ti, 1) == g["total"]["speedup"]
    # Table 2's F_l column is the fragment count entering each conv layer
    ext = ix.fragment_extents(wl.n4_layers(), 512, 512)
    assert [len(ext[l - 1]) for l in (1, 3, 5, 7)] == [r[7] for r in g["rows"]]


# ---- Hand evaluation (Sections 2.1.1, 2.1.2, softmax of Section 1) --------

def test_hand_ramp_boxsum_pool():
    case = _gold("hand_cases.json")["cases"][0]
    img = (10.0 * np.arange(5)[:, None] + np.arange(5)[None, :]).reshape(1, 5, 5, 1)
    layers = [wl.conv(2, 1, 1, "none"), wl.pool(2, 1), wl.fc(1, 1, 1, "none")]
    params = [(np.ones((1, 1, 2, 2)), np.zeros(1)), None, (np.ones((1, 1, 1, 1)), np.zeros(1))]
    out = oracle.patch_forward(layers, params, img, 3)
    assert np.array_equal(out[0, :, :, 0], np.array(case["expected"], np.float64))


def test_hand_impulse_tanh():
    img = np.zeros((1, 4, 4, 1))
    img[0, 2, 1, 0] = 1.0
    w = np.array([[0.5, -1.0], [2.0, 0.25]])
    layers = [wl.conv(2, 1, 1, "tanh"), wl.fc(2, 1, 1, "none")]
    params = [(w.reshape(1, 1, 2, 2), np.array([0.1])), (np.ones((1, 1, 2, 2)), np.zeros(1))]
    out = oracle.patch_forward(layers, params, img, 3)
    for Y in range(2):
        for X in range(2):
            s = 0.0
            for y in range(2):
                for x in range(2):
                    i, j = 2 - Y - y, 1 - X - x
                    s += math.tanh(0.1 + (w[i, j] if 0 <= i <= 1 and 0 <= j <= 1 else 0.0))
            assert out[0, Y, X, 0] == pytest.approx(s, abs=1e-15)


def test_hand_softmax_two_class():
    img = (np.arange(2)[:, None] + 2.0 * np.arange(2)[None, :]).reshape(1, 2, 2, 1)
    layers = [wl.fc(1, 1, 2, "softmax")]
    params = [(np.array([1.0, -1.0]).reshape(2, 1, 1, 1), np.array([0.0, 0.5]))]
    out = oracle.patch_forward(layers, params, img, 1)
    for Y in range(2):
        for X in range(2):
            v = Y + 2.0 * X
            p0 = 1.0 / (1.0 + math.exp(-2 * v + 0.5))
            assert out[0, Y, X, 0] == pytest.approx(p0, abs=1e-15)
            assert out[0, Y, X, 1] == pytest.approx(1 - p0, abs=1e-15)


# ---- Library special cases -------------------------------------------------

@pytest.mark.parametrize("wid", [1, 2, 3, 5])
def test_single_patch_equals_library_net(wid):
    """H = W = w_0: one patch, where the scan is the plain net; torch CPU
    conv2d / max_pool2d / linear / softmax in float64."""
    w = wl.WORKLOADS[wid]
    params, _ = wl.workload_inputs(wid)
    img = wl.make_image(7, 1, w.patch, w.patch, w.channels)
    got = oracle.patch_forward(w.layers, params, img, w.patch)[0, 0, 0]
    want = torch_patch_net(w.layers, params, img[0])
    assert np.abs(got - want).max() <= 1e-12


def test_single_patch_random_nets():
    for seed in range(15):
        rng = np.random.default_rng(500 + seed)
        layers, w0, c0 = wl.random_net(rng)
        params = wl.make_weights(layers, seed, 0.5)
        img = wl.make_image(seed, 1, w0, w0, c0)
        got = oracle.patch_forward(layers, params, img, w0)[0, 0, 0]
        want = torch_patch_net(layers, params, img[0])
        assert np.abs(got - want).max() <= 1e-12, seed


def test_no_pool_net_is_whole_image_conv():
    """Section 1: without pooling the scan is the plain convolutions applied
    to the entire image (torch CPU conv2d on the full image)."""
    import torch
    import torch.nn.functional as F
    layers = [wl.conv(3, 2, 5), wl.conv(2, 5, 4), wl.fc(3, 4, 3, "none")]
    params = wl.make_weights(layers, 11, 0.4)
    img = wl.make_image(12, 2, 17, 13, 2)
    got = oracle.patch_forward(layers, params, img, 6)
    x = torch.from_numpy(img.astype(np.float64)).permute(0, 3, 1, 2)
    for L, (w, b) in zip(layers, params):
        x = F.conv2d(x, torch.from_numpy(w.astype(np.float64)), torch.from_numpy(b.astype(np.float64)))
        if L["act"] == "tanh":
            x = torch.tanh(x)
    want = x.permute(0, 2, 3, 1).numpy()
    assert got.shape == want.shape
    assert np.abs(got - want).max() <= 1e-12


@pytest.mark.parametrize("seed", range(12))
def test_dilated_whole_map(seed):
    rng = np.random.default_rng(900 + seed)
    layers, w0, c0 = wl.random_net(rng)
    params = wl.make_weights(layers, seed, 0.5)
    H = w0 + int(rng.integers(0, 11))
    W = w0 + int(rng.integers(0, 11))
    img = wl.make_image(seed, 2, H, W, c0)
    got = oracle.patch_forward(layers, params, img, w0)
    want = dilated_scan(layers, params, img)
    assert got.shape == want.shape
    assert np.abs(got - want).max() <= 1e-12


# ---- Exactness: the fragment method equals the per-patch definition --------

@pytest.mark.parametrize("seed", range(25))
def test_frag_cpu_equals_patch_oracle(seed):
    """Fig. 2's caption: the image-based method is exact, so the fragment
    computation on the CPU gives the per-patch outputs."""
    rng = np.random.default_rng(300 + seed)
    layers, w0, c0 = wl.random_net(rng)
    params = wl.make_weights(layers, seed, 0.5)
    H = w0 + int(rng.integers(0, 15))
    W = w0 + int(rng.integers(0, 15))
    B = int(rng.integers(1, 3))
    img = wl.make_image(seed, B, H, W, c0)
    ref = oracle.patch_forward(layers, params, img, w0)
    got = oracle.frag_cpu.frag_scan(layers, params, img, w0)
    assert not np.isnan(got).any()
    assert np.abs(got - ref).max() <= 1e-12


def test_frag_cpu_workload1_full():
    w = wl.WORKLOADS[1]
    params, img = wl.workload_inputs(1)
    ref = oracle.patch_forward(w.layers, params, img, w.patch)
    got = oracle.frag_cpu.frag_scan(w.layers, params, img, w.patch)
    assert np.abs(got - ref).max() <= 1e-12


def test_frag_cpu_workload5_net_sample():
    """Workload 5's net (3x3 pool) on a 100 x 90 image, sampled patches."""
    w = wl.WORKLOADS[5]
    params, _ = wl.workload_inputs(5)
    img = wl.make_image(105, 1, 100, 90, 3)
    got = oracle.frag_cpu.frag_scan(w.layers, params, img, w.patch)
    rng = np.random.default_rng(0)
    pts = np.stack([np.zeros(64, int), rng.integers(0, 40, 64), rng.integers(0, 30, 64)], 1)
    ref = oracle.patch_forward(w.layers, params, img, w.patch, pts)
    assert np.abs(got[0, pts[:, 1], pts[:, 2]] - ref).max() <= 1e-12


# ---- Rectangular kernels and pools (Section 2: the square case generalizes
# ---- directly; every rule holds per axis) -----------------------------------

@pytest.mark.parametrize("seed", range(16))
def test_rect_sizes_counts_and_coverage(seed):
    rng = np.random.default_rng(1500 + seed)
    layers, (h0, w0), _ = wl.random_rect_net(rng)
    assert ix.patch_hw(layers) == (h0, w0)
    assert ix.patch_sizes(layers, h0, 0)[-1] == 1 == ix.patch_sizes(layers, w0, 1)[-1]
    prod = 1
    for L in layers:
        if L["kind"] == "pool":
            prod *= L["k"] * L.get("kx", L["k"])
    H, W = h0 + int(rng.integers(0, 11)), w0 + int(rng.integers(0, 11))
    ext = ix.fragment_extents(layers, H, W)
    assert len(ext[-1]) == prod == ix.n_fragments(layers)
    for frags in ext:
        ys, xs = [e[0] for e in frags], [e[1] for e in frags]
        assert max(ys) - min(ys) <= 1 and max(xs) - min(xs) <= 1
    idx = ix.reassembly_index(layers, H, W).reshape(-1, 3)
    keys = set(map(tuple, idx.tolist()))
    assert len(keys) == idx.shape[0] == (H - h0 + 1) * (W - w0 + 1)
    assert sum(a * b for a, b in ext[-1]) == len(keys)
    for f, e in ix.fragment_table(layers, H, W).items():
        assert e["size"] == ext[-1][f]


@pytest.mark.parametrize("seed", range(10))
def test_rect_window_equals_library_net(seed):
    rng = np.random.default_rng(1600 + seed)
    layers, (h0, w0), c0 = wl.random_rect_net(rng)
    params = wl.make_weights(layers, seed, 0.5)
    img = wl.make_image(seed, 1, h0, w0, c0)
    got = oracle.patch_forward(layers, params, img, (h0, w0))[0, 0, 0]
    assert np.abs(got - torch_patch_net(layers, params, img[0])).max() <= 1e-12


@pytest.mark.parametrize("seed", range(10))
def test_rect_whole_map_and_frag_cpu(seed):
    """Whole map == the dilated library formulation, and the fragment method
    on the CPU == the per-window definition, with rectangular layers."""
    rng = np.random.default_rng(1700 + seed)
    layers, (h0, w0), c0 = wl.random_rect_net(rng)
    params = wl.make_weights(layers, seed, 0.5)
    img = wl.make_image(seed, 2, h0 + int(rng.integers(0, 9)), w0 + int(rng.integers(0, 9)), c0)
    ref = oracle.patch_forward(layers, params, img, (h0, w0))
    assert np.abs(ref - dilated_scan(layers, params, img)).max() <= 1e-12
    got = oracle.frag_cpu.frag_scan(layers, params, img, (h0, w0))
    assert not np.isnan(got).any()
    assert np.abs(got - ref).max() <= 1e-12


# ---- Pools whose stride differs from their size (a generalisation: the
# ---- paper's pools do not overlap, Section 2.1.2) ---------------------------

def test_hand_stride_pools():
    """Overlapping (3x3, stride 2) and gapped (2x2, stride 3) pools on a
    ramp: closed forms worked out by hand, for the per-window oracle and the
    CPU fragment method."""
    g = _gold("hand_stride_pools.json")
    img = (10.0 * np.arange(7)[:, None] + np.arange(6)[None, :]).reshape(1, 7, 6, 1)
    for case in g["cases"]:
        k, st = case["pool"]["k"], case["pool"]["stride"]
        layers = [wl.pool(k, 1, stride=st), wl.fc(2, 1, 1, "none")]
        params = [None, (np.ones((1, 1, 2, 2)), np.zeros(1))]
        assert ix.patch_size(layers) == 5
        want = np.array(case["expected"], np.float64)
        assert np.array_equal(oracle.patch_forward(layers, params, img, 5)[0, :, :, 0], want), case["name"]
        assert np.array_equal(oracle.frag_cpu.frag_scan(layers, params, img, 5)[0, :, :, 0], want), case["name"]


def test_stride_equal_to_size_is_the_paper_pool():
    """A stride equal to the pool's size changes nothing: the same sizes,
    fragments and outputs as the plain pool of Section 2.2.2."""
    plain = wl.WORKLOADS[1].layers
    strided = [dict(L, stride=L["k"], stride_x=L["k"]) if L["kind"] == "pool" else L for L in plain]
    params, img = wl.workload_inputs(1, height=30, width=27)
    assert ix.fragment_extents(plain, 30, 27) == ix.fragment_extents(strided, 30, 27)
    assert np.array_equal(ix.reassembly_index(plain, 30, 27), ix.reassembly_index(strided, 30, 27))
    assert np.array_equal(oracle.patch_forward(plain, params, img, 14), oracle.patch_forward(strided, params, img, 14))


@pytest.mark.parametrize("seed", range(16))
def test_stride_sizes_counts_and_coverage(seed):
    """Random stacks with overlapping and gapped pools: the window derived
    bottom-up reduces to 1 x 1, there are prod(s_y * s_x) final fragments,
    and every window lands on exactly one position of one final fragment
    (corner tracking), inside the fragment sizes of the extent recursion."""
    rng = np.random.default_rng(2500 + seed)
    layers, (h0, w0), _ = wl.random_stride_net(rng)
    assert ix.patch_hw(layers) == (h0, w0)
    assert ix.patch_sizes(layers, h0, 0)[-1] == 1 == ix.patch_sizes(layers, w0, 1)[-1]
    prod = 1
    for L in layers:
        if L["kind"] == "pool":
            prod *= ix.syx(L)[0] * ix.syx(L)[1]
    H, W = h0 + int(rng.integers(0, 15)), w0 + int(rng.integers(0, 15))
    ext = ix.fragment_extents(layers, H, W)
    assert len(ext[-1]) == prod == ix.n_fragments(layers)
    idx = ix.reassembly_index(layers, H, W).reshape(-1, 3)
    keys = set(map(tuple, idx.tolist()))
    assert len(keys) == idx.shape[0] == (H - h0 + 1) * (W - w0 + 1)
    assert sum(a * b for a, b in ext[-1]) == len(keys)
    for f, e in ix.fragment_table(layers, H, W).items():
        assert e["size"] == ext[-1][f]


@pytest.mark.parametrize("seed", range(10))
def test_stride_window_equals_library_net(seed):
    """One window == torch's max_pool2d with the same stride (library
    routine) in a torch-CPU net."""
    rng = np.random.default_rng(2600 + seed)
    layers, (h0, w0), c0 = wl.random_stride_net(rng)
    params = wl.make_weights(layers, seed, 0.5)
    img = wl.make_image(seed, 1, h0, w0, c0)
    got = oracle.patch_forward(layers, params, img, (h0, w0))[0, 0, 0]
    assert np.abs(got - torch_patch_net(layers, params, img[0])).max() <= 1e-12


@pytest.mark.parametrize("seed", range(10))
def test_stride_whole_map_and_frag_cpu(seed):
    """Whole map == the dilated library formulation (a pool of stride s
    multiplies the dilation by s), and the CPU fragment method == the
    per-window definition, with overlapping and gapped pools."""
    rng = np.random.default_rng(2700 + seed)
    layers, (h0, w0), c0 = wl.random_stride_net(rng)
    params = wl.make_weights(layers, seed, 0.5)
    img = wl.make_image(seed, 2, h0 + int(rng.integers(0, 9)), w0 + int(rng.integers(0, 9)), c0)
    ref = oracle.patch_forward(layers, params, img, (h0, w0))
    assert np.abs(ref - dilated_scan(layers, params, img)).max() <= 1e-12
    got = oracle.frag_cpu.frag_scan(layers, params, img, (h0, w0))
    assert not np.isnan(got).any()
    assert np.abs(got - ref).max() <= 1e-12
