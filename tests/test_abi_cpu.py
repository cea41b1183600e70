"""Host-side checks of the C-ABI library (no GPU needed).

The library must load and export every entry point include/fragscan.h
declares; its host planner (fragment sizes, fragment table, reassembly index,
work counts) must agree bit for bit with the oracle's independent index code;
and its argument checks must reject bad input before any device work.
"""
import ctypes
import os
import re

import numpy as np
import pytest

from oracle import index as ix
from paper_1302_1700_amd import fragscan as fsb
from paper_1302_1700_amd import workloads as wl

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _header_functions():
    src = open(os.path.join(ROOT, "include", "fragscan.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(fs_[a-z_]+)\s*\(", src)))


def test_library_exports_every_declared_function():
    lib = fsb.load()
    names = _header_functions()
    assert "fs_scan" in names and "fs_net_create" in names
    for n in names:
        assert hasattr(lib, n), n
    assert set(names) == set(fsb.EXPORTS)


def _plan_net(layers, params=None, c0=1, patch=0, dtype="f32"):
    if params is None:
        params = wl.make_weights(layers, 0, 0.1)
    return fsb.Net(layers, params, c0, patch, dtype, plan_only=True)


def _check_tables(layers, H, W, c0=1):
    net = _plan_net(layers, c0=c0)
    h0, w0 = ix.patch_hw(layers)
    assert (net.patch, net.patch_x) == (h0, w0)
    Sy = Sx = 1
    for L in layers:
        if L["kind"] == "pool":
            Sy, Sx = Sy * ix.syx(L)[0], Sx * ix.syx(L)[1]
    assert (net.info["stride"], net.info["stride_x"]) == (Sy, Sx)
    assert net.info["n_fragments"] == ix.n_fragments(layers)
    # reassembly index, every output pixel
    got = net.reassembly_index(H, W)
    want = ix.reassembly_index(layers, H, W)
    assert got.shape == want.shape
    assert np.array_equal(got, want.astype(np.int32))
    # fragment table
    tab = net.fragment_table(H, W)
    F = ix.n_fragments(layers)
    assert tab.shape[0] == F
    assert np.array_equal(tab[:, 0], np.arange(F))
    ext = ix.fragment_extents(layers, H, W)[-1]
    want_tab = ix.fragment_table(layers, H, W)
    for row in tab:
        f, h, w, Y0, X0 = (int(v) for v in row[:5])
        assert (h, w) == ext[f]
        if f in want_tab:
            e = want_tab[f]
            assert (h, w) == e["size"]
            assert (Y0, X0) == e["base"]
            offs = [(int(row[5 + 2 * m]), int(row[6 + 2 * m])) for m in range(len(e["offsets"]))]
            assert offs == e["offsets"]
        else:
            assert h * w == 0
    # plan: output size and algorithmic FLOPs
    p = net.plan(2, H, W)
    assert (p["out_h"], p["out_w"]) == (H - h0 + 1, W - w0 + 1)
    assert p["flops"] == pytest.approx(sum(ix.algorithmic_flops(layers, 2, H, W)), rel=1e-12)
    net.close()


@pytest.mark.parametrize("wid", [1, 2, 3, 5])
def test_tables_workload_nets(wid):
    w = wl.WORKLOADS[wid]
    H = {1: 64, 2: 160, 3: 190, 5: 130}[wid]
    _check_tables(w.layers, H, H + 7, w.channels)


def test_tables_workload_full_sizes():
    """Full-size workloads: sizes and work counts against the oracle's index
    code (the per-pixel tables are compared on the smaller images above)."""
    for wid, w in wl.WORKLOADS.items():
        net = _plan_net(w.layers, c0=w.channels, dtype=w.dtype)
        p = net.plan(w.batch, w.height, w.width)
        assert p["out_h"] == w.out_h and p["out_w"] == w.out_w
        assert p["flops"] == pytest.approx(sum(ix.algorithmic_flops(w.layers, w.batch, w.height, w.width)),
                                           rel=1e-12)
        ri = net.reassembly_index(w.height, w.width)
        want = ix.reassembly_index(w.layers, w.height, w.width)
        assert np.array_equal(ri, want.astype(np.int32))
        net.close()


@pytest.mark.parametrize("seed", range(25))
def test_tables_random_nets(seed):
    rng = np.random.default_rng(4000 + seed)
    layers, w0, c0 = wl.random_net(rng)
    H = w0 + int(rng.integers(0, 20))
    W = w0 + int(rng.integers(0, 20))
    _check_tables(layers, H, W, c0)


@pytest.mark.parametrize("seed", range(25))
def test_tables_random_rect_nets(seed):
    """Rectangular kernels and pools (Section 2: every rule per axis)."""
    rng = np.random.default_rng(4500 + seed)
    layers, (h0, w0), c0 = wl.random_rect_net(rng)
    H = h0 + int(rng.integers(0, 20))
    W = w0 + int(rng.integers(0, 20))
    _check_tables(layers, H, W, c0)


def test_rect_net_rules():
    """A 2 x 3 pool gives 6 children (f * 6 + o_y * 3 + o_x); the window is
    derived per axis; a square patch argument or a k_x on an FC layer that
    takes its size from the map is rejected."""
    layers = [wl.conv(2, 1, 2, "tanh", kx=3), wl.pool(2, 2, kx=3), wl.fc(2, 2, 3, "tanh", kx=1),
              wl.fc(1, 3, 2, "softmax")]
    net = _plan_net(layers)
    assert (net.patch, net.patch_x) == (5, 5)
    assert net.info["n_fragments"] == 6 and (net.info["stride"], net.info["stride_x"]) == (2, 3)
    tab = net.fragment_table(12, 15)
    assert [tuple(r[5:7]) for r in tab] == [(ox, oy) for oy in range(2) for ox in range(3)]
    net.close()
    layers = [wl.conv(3, 1, 2, "tanh", kx=1), wl.pool(1, 2, kx=2), wl.fc(2, 2, 2, "softmax", kx=3)]
    assert ix.patch_hw(layers) == (4, 6)
    net = _plan_net(layers)
    assert (net.patch, net.patch_x) == (4, 6)
    assert net.plan(1, 10, 20)["out_h"] == 7 and net.plan(1, 10, 20)["out_w"] == 15
    with pytest.raises(fsb.FsError):
        net.plan(1, 10, 5)  # narrower than w_0 = 6
    net.close()
    assert _status(layers, patch=4) == fsb.FS_ERR_SHAPE
    assert _status(layers, patch=6) == fsb.FS_ERR_SHAPE
    bad = [dict(L) for L in layers]
    bad[-1]["k"], bad[-1]["kx"] = 0, 3
    params = wl.make_weights(layers, 0, 0.1)
    assert _status(bad, params, patch=4) == fsb.FS_ERR_SHAPE
    # a 2 x 3 pool on a map whose columns it does not divide (5 x 5 window,
    # 4 x 4 map after the convolution)
    bad = [wl.conv(2, 1, 2, "tanh"), wl.pool(2, 2, kx=3), wl.fc(0, 2, 2, "softmax")]
    params = [(np.zeros((2, 1, 2, 2), np.float32), None), None, (np.zeros((2, 2, 3, 2), np.float32), None)]
    assert _status(bad, params, patch=5) == fsb.FS_ERR_SHAPE
    # 6 x 6 map: 3 x 2 after the pool, and the last layer takes a 3 x 2 kernel
    assert _status(bad, params, patch=7) == fsb.FS_OK


def test_single_window_image():
    """H = W = w_0: one output; all final fragments but one are empty."""
    _check_tables(wl.WORKLOADS[2].layers, 95, 95)


# ---- error paths (checked before any device work) ---------------------------

def _status(layers, params=None, c0=1, patch=0, dtype="f32"):
    try:
        _plan_net(layers, params, c0, patch, dtype).close()
        return fsb.FS_OK
    except fsb.FsError as e:
        return e.status


def test_rejects_bad_nets():
    # pool that does not divide the patch-level map (Section 2.1.2)
    assert _status([wl.conv(2, 1, 2), wl.pool(2, 2), wl.fc(2, 2, 2)], patch=6) == fsb.FS_ERR_SHAPE
    # workload 5 with its stated patch of 57: its 3x3 pool would see a 53 map
    w5 = wl.WORKLOADS[5]
    params5, _ = wl.workload_inputs(5, height=61, width=61)
    assert _status(w5.layers, params5, 3, 57, "bf16") == fsb.FS_ERR_SHAPE
    assert _status(w5.layers, params5, 3, 61, "bf16") == fsb.FS_OK
    # channel mismatch
    assert _status([wl.conv(2, 1, 3), wl.fc(2, 4, 2)]) == fsb.FS_ERR_SHAPE
    # softmax before the last layer
    assert _status([wl.conv(2, 1, 3, "softmax"), wl.fc(2, 3, 2)]) == fsb.FS_ERR_SHAPE
    # last map not 1x1
    assert _status([wl.conv(2, 1, 3), wl.fc(2, 3, 2)], patch=5) == fsb.FS_ERR_SHAPE
    # convolution after a fully connected layer
    assert _status([wl.fc(2, 1, 3), wl.conv(1, 3, 2)]) == fsb.FS_ERR_SHAPE
    # more classes than the head supports
    assert _status([wl.fc(2, 1, 17)]) == fsb.FS_ERR_UNSUPPORTED
    # a net without pools is the plain whole-image case (Section 1)
    assert _status([wl.conv(2, 1, 2, "none"), wl.fc(1, 2, 2)]) == fsb.FS_OK


def test_split_k_needs_a_step_per_wave(monkeypatch):
    # a 1x1 16 -> 16 layer has one K step; forcing two K-splitting waves on
    # it (tuning override) is refused instead of leaving a wave without work
    layers = [wl.conv(1, 16, 16), wl.fc(1, 16, 2, "softmax")]
    monkeypatch.setenv("FRAGSCAN_TILE", "0:0,0,0,0,2")
    assert _status(layers, c0=16) == fsb.FS_ERR_UNSUPPORTED
    monkeypatch.delenv("FRAGSCAN_TILE")
    assert _status(layers, c0=16) == fsb.FS_OK


def test_border_plans():
    """Mirrored borders (Section 3.2): H x W outputs for any H, W >= 1, the
    scan of the extended image plus room for it in the workspace."""
    w = wl.WORKLOADS[2]
    net = _plan_net(w.layers)
    for mode in ("reflect", "symmetric"):
        for H, W in ((512, 512), (40, 33), (1, 1)):
            p = net.plan(1, H, W, mode)
            assert (p["out_h"], p["out_w"]) == (H, W)
            inner = net.plan(1, H + w.patch - 1, W + w.patch - 1)
            assert p["workspace_bytes"] >= inner["workspace_bytes"] + (H + w.patch - 1) * (W + w.patch - 1) * 4
            assert p["n_launches"] == inner["n_launches"] + 1
    assert net.plan(2, 512, 512, "valid") == net.plan(2, 512, 512)
    net.close()


RUN_NET = [wl.conv(3, 3, 32), wl.conv(2, 32, 64), wl.pool(2, 64), wl.conv(2, 64, 40),
           wl.conv(1, 40, 18), wl.pool(2, 18), wl.fc(2, 18, 24), wl.fc(1, 24, 3, "softmax")]


@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_run_tile_plans(monkeypatch, dt):
    """One-band layers whose fragments all hold a tile's worth of outputs
    can take run tiles (named +run): the split-K vector layer at the smaller
    image, the gather layer with the fused head at the larger one (pools not
    fused); FRAGSCAN_RUN=1 keeps them wherever they fit, =0 turns them off,
    and a run launch needs no more workgroups than per-fragment tiles."""
    w0 = ix.patch_size(RUN_NET)
    cases = (((w0 + 41, w0 + 29), "", {3}), ((w0 + 90, w0 + 77), "0", {6}))
    for (H, W), fuse, want in cases:
        monkeypatch.setenv("FRAGSCAN_POOL_FUSE", fuse)
        monkeypatch.setenv("FRAGSCAN_RUN", "1")
        net = _plan_net(RUN_NET, c0=3, dtype=dt)
        on = net.launches(2, H, W)
        monkeypatch.setenv("FRAGSCAN_RUN", "0")
        off = net.launches(2, H, W)
        net.close()
        assert {L["layer"] for L in on if L["name"].endswith("+run")} == want
        assert not any("+run" in L["name"] for L in off)
        for a, b in zip(on, off):
            assert a["out_pixels"] == b["out_pixels"] and a["flops"] == b["flops"]
            if a["layer"] in want:
                assert a["grid"] <= b["grid"]


def test_run_tiles_where_they_save_a_round(monkeypatch):
    """By default run tiles are kept only where they need fewer rounds of
    workgroups (plan-only nets count 256 CUs, one workgroup each): N4's 3x3
    layer with the fused head on 448 x 448 (1280 per-fragment tiles, 980 run
    tiles) but not on 512 x 512 (1536 against 1375: six rounds either way)."""
    monkeypatch.delenv("FRAGSCAN_RUN", raising=False)
    net = _plan_net(wl.WORKLOADS[2].layers)
    fc = {H: [L for L in net.launches(1, H, H) if L["layer"] == 8][0] for H in (448, 512)}
    net.close()
    assert fc[448]["name"].endswith("+head+run") and fc[448]["grid"] == 984
    assert fc[512]["name"].endswith("+head") and fc[512]["grid"] == 1536


def test_row_tiles_where_one_workgroup_per_cu(monkeypatch):
    """N4's 5x5 layer on a 494 x 494 image: 16-column bands leave a 2-column
    last band, whose 128-pixel tiles span 64 rows; sized for those, the LDS
    would admit one workgroup per CU, so the planner takes tiles of 8 whole
    band rows (plan-only nets count LDS only).  FRAGSCAN_ROWTILES=0/1 forces
    either; at 512 x 512 (last band 10 columns) pixel tiles fit three per CU
    and stay."""
    monkeypatch.delenv("FRAGSCAN_ROWTILES", raising=False)
    net = _plan_net(wl.WORKLOADS[2].layers)
    conv5 = lambda H: [L for L in net.launches(1, H, H) if L["layer"] == 2][0]
    auto = conv5(494)
    monkeypatch.setenv("FRAGSCAN_ROWTILES", "0")
    pix = conv5(494)
    pix512 = conv5(512)
    monkeypatch.setenv("FRAGSCAN_ROWTILES", "1")
    rows = conv5(494)
    monkeypatch.delenv("FRAGSCAN_ROWTILES")
    at512 = conv5(512)
    net.close()
    assert pix["lds_bytes"] > 160 * 1024 // 2 >= rows["lds_bytes"]
    assert auto["lds_bytes"] == rows["lds_bytes"] and auto["grid"] == rows["grid"]
    assert at512["lds_bytes"] == pix512["lds_bytes"] <= 160 * 1024 // 3
    assert auto["out_pixels"] == pix["out_pixels"] == rows["out_pixels"]


def test_wide_fc_tile_plan(monkeypatch):
    """The float32 4 x 13 tile for a 200-output FC layer with the fused head:
    forced on, one 256-pixel tile per workgroup and a single channel-block
    group; forced off, the 7 x 2 tiles."""
    w = wl.WORKLOADS[2]
    names = {}
    for mode in ("1", "0"):
        monkeypatch.setenv("FRAGSCAN_WIDE", mode)
        net = _plan_net(w.layers, c0=w.channels)
        fc = [L for L in net.launches(1, w.height, w.width) if L["name"].endswith("+head")][0]
        names[mode] = fc
        net.close()
    assert names["1"]["name"].startswith("conv_frag_mfma<4, 13, 1, 1, false")
    assert names["0"]["name"].startswith("conv_frag_mfma<4, 7, 2, 1, false")
    assert names["1"]["grid"] * 2 == names["0"]["grid"]  # 256- against 128-pixel tiles
    assert names["1"]["flops"] == names["0"]["flops"]
    # bf16 nets and other channel counts keep their tiles
    monkeypatch.setenv("FRAGSCAN_WIDE", "1")
    net = _plan_net(w.layers, c0=w.channels, dtype="bf16")
    assert all("<4, 13," not in L["name"] for L in net.launches(1, w.height, w.width))
    net.close()


def test_tiled_plans():
    """Tiled scan plans: the same output map, a workspace bounded by the
    tile, one scan's launches per tile, and the halo recomputed (more FLOPs
    than one scan, the same for a tile covering the map)."""
    w = wl.WORKLOADS[2]
    net = _plan_net(w.layers)
    full = net.plan(2, 700, 650)
    ny, nx = full["out_h"], full["out_w"]
    for th, tw in ((128, 96), (1, 1000), (ny, nx), (ny + 5, nx + 9)):
        t = net.plan_tiled(2, 700, 650, (th, tw))
        assert (t["out_h"], t["out_w"]) == (ny, nx)
        rows, cols = -(-ny // min(th, ny)), -(-nx // min(tw, nx))
        assert t["n_launches"] == rows * cols * full["n_launches"]
        if rows * cols == 1:
            assert t["workspace_bytes"] == full["workspace_bytes"] and t["flops"] == full["flops"]
        else:
            assert t["workspace_bytes"] < full["workspace_bytes"] and t["flops"] > full["flops"]
    for bad in ((0, 5), (5, 0)):
        with pytest.raises(fsb.FsError) as e:
            net.plan_tiled(1, 200, 200, bad)
        assert e.value.status == fsb.FS_ERR_INVALID_ARG
    net.close()
    # a net that starts with a pool reads the image with the fragment kernels'
    # own pitch: not tiled
    layers = [wl.pool(2, 1), wl.conv(3, 1, 4), wl.fc(1, 4, 2, "softmax")]
    net = _plan_net(layers)
    with pytest.raises(fsb.FsError) as e:
        net.plan_tiled(1, 40, 40, (8, 8))
    assert e.value.status == fsb.FS_ERR_UNSUPPORTED
    net.close()


def test_border_mode_rejected_when_unknown():
    net = _plan_net(wl.WORKLOADS[1].layers)
    p = fsb.fs_plan_info()
    st = fsb.load().fs_scan_plan_border(net._h, 1, 64, 64, 7, fsb.ctypes.byref(p))
    assert st == fsb.FS_ERR_INVALID_ARG
    net.close()


def test_image_smaller_than_patch_rejected():
    net = _plan_net(wl.WORKLOADS[1].layers)
    with pytest.raises(fsb.FsError) as e:
        net.plan(1, 13, 64)
    assert e.value.status == fsb.FS_ERR_SHAPE
    net.close()


def test_scan_argument_checks_without_device():
    lib = fsb.load()
    net = _plan_net(wl.WORKLOADS[1].layers)
    p = net.plan(1, 64, 64)
    img, out, ws = ctypes.c_void_p(1 << 20), ctypes.c_void_p(2 << 20), ctypes.c_void_p(4 << 20)
    st = lib.fs_scan(net._h, img, 1, 64, 64, out, ws, p["workspace_bytes"] - 1, None)
    assert st == fsb.FS_ERR_WORKSPACE
    st = lib.fs_scan(net._h, ctypes.c_void_p((1 << 20) + 4), 1, 64, 64, out, ws, p["workspace_bytes"], None)
    assert st == fsb.FS_ERR_INVALID_ARG
    st = lib.fs_scan(net._h, img, 1, 64, 64, out, ctypes.c_void_p((4 << 20) + 16), p["workspace_bytes"], None)
    assert st == fsb.FS_ERR_INVALID_ARG
    st = lib.fs_scan(net._h, None, 1, 64, 64, out, ws, p["workspace_bytes"], None)
    assert st == fsb.FS_ERR_INVALID_ARG
    st = lib.fs_scan(net._h, img, 1, 10, 64, out, ws, p["workspace_bytes"], None)
    assert st == fsb.FS_ERR_SHAPE
    # a planning-only net never launches
    st = lib.fs_scan(net._h, img, 1, 64, 64, out, ws, p["workspace_bytes"], None)
    assert st == fsb.FS_ERR_INVALID_ARG
    assert b"planning only" in lib.fs_last_error()
    net.close()


def test_status_strings():
    for debug in (False, True):
        lib = fsb.load(debug)
        strs = [lib.fs_status_str(s) for s in range(fsb.FS_ERR_BOUNDS + 1)]
        assert all(strs) and len(set(strs)) == len(strs)
        assert b"bounds" in strs[fsb.FS_ERR_BOUNDS]


def test_debug_library_exports_and_plans():
    """libfragscan_debug.so (the same sources with the kernels' bounds checks
    compiled in) exports every declared entry point and plans the workload
    nets and random nets launch for launch as the release library does."""
    lib = fsb.load(debug=True)
    for n in _header_functions():
        assert hasattr(lib, n), n
    cases = [(w.layers, w.channels, w.dtype, w.batch, w.height, w.width) for w in wl.WORKLOADS.values()]
    for seed in range(6):
        rng = np.random.default_rng(400 + seed)
        layers, w0, c0 = wl.random_net(rng, max_c=40)
        cases.append((layers, c0, "bf16" if seed % 2 else "f32", 2, w0 + 37, w0 + 23))
    for layers, c0, dt, B, H, W in cases:
        params = wl.make_weights(layers, 0, 0.1)
        plans = []
        for debug in (False, True):
            net = fsb.Net(layers, params, c0, 0, dt, plan_only=True, debug=debug)
            plans.append((net.plan(B, H, W), net.launches(B, H, W)))
            net.close()
        assert plans[0] == plans[1]


def test_bench_cpu_fragment_leg():
    """bench.py's CPU fragment leg: the full image when it is small enough, a
    top-left crop of image 0 with the requested number of windows otherwise,
    and a crop scan that gives the full scan's values on those windows."""
    import sys
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    sys.path.insert(0, root)
    import bench
    import oracle
    w = wl.WORKLOADS[1]
    params, img = wl.workload_inputs(1)
    full = bench.cpu_fragment_baseline(w, params, img)
    assert full["sample"] == "full image" and full["value"] > 0
    crop = bench.cpu_fragment_baseline(w, params, img, max_windows=144)
    assert crop["sample"] == "top-left crop 25x25 of image 0 (144 windows)", crop["sample"]
    whole = oracle.frag_cpu.frag_scan(w.layers, params, img, w.patch)
    part = oracle.frag_cpu.frag_scan(w.layers, params, img[:1, :25, :25], w.patch)
    assert part.shape == (1, 12, 12, w.n_classes)
    assert np.abs(part - whole[:1, :12, :12]).max() <= 1e-12


def test_misaligned_pointers_named_in_error():
    """The alignment contract of fs_scan (16-byte image and output, 256-byte
    workspace), checked before anything else touches the pointers."""
    lib = fsb.load()
    net = _plan_net(wl.WORKLOADS[1].layers)
    n = net.plan(1, 64, 64)["workspace_bytes"]
    img, out, ws = ctypes.c_void_p(1 << 20), ctypes.c_void_p(2 << 20), ctypes.c_void_p(4 << 20)
    for bad_img, bad_out in (((1 << 20) + 8, 2 << 20), (1 << 20, (2 << 20) + 4)):
        st = lib.fs_scan(net._h, ctypes.c_void_p(bad_img), 1, 64, 64, ctypes.c_void_p(bad_out), ws, n, None)
        assert st == fsb.FS_ERR_INVALID_ARG and b"16-byte" in lib.fs_last_error()
    # 16 bytes is enough for the image and output; the workspace needs 256
    st = lib.fs_scan(net._h, ctypes.c_void_p((1 << 20) + 16), 1, 64, 64, ctypes.c_void_p((2 << 20) + 48),
                     ctypes.c_void_p((4 << 20) + 128), n, None)
    assert st == fsb.FS_ERR_INVALID_ARG and b"256-byte" in lib.fs_last_error()
    for fn, extra in ((lib.fs_scan_border, (1,)), ):
        st = fn(net._h, ctypes.c_void_p((1 << 20) + 4), 1, 64, 64, *extra, out, ws, 1 << 30, None)
        assert st == fsb.FS_ERR_INVALID_ARG and b"16-byte" in lib.fs_last_error()
    st = lib.fs_scan_tiled(net._h, ctypes.c_void_p((1 << 20) + 4), 1, 64, 64, 8, 8, out, ws, 1 << 30, None)
    assert st == fsb.FS_ERR_INVALID_ARG and b"16-byte" in lib.fs_last_error()
    net.close()


def test_image_side_limit():
    """Fragment sizes travel in 16-bit tables: an image side above 65535 is
    refused (not scanned wrongly), and the tiled scan takes such an image in
    regions below the limit."""
    net = _plan_net(wl.WORKLOADS[1].layers)
    assert net.plan(1, 64, 65535)["out_w"] == 65535 - 14 + 1
    for H, W in ((64, 65536), (65536, 64), (64, 70000)):
        with pytest.raises(fsb.FsError) as e:
            net.plan(1, H, W)
        assert e.value.status == fsb.FS_ERR_UNSUPPORTED and "fs_scan_tiled" in str(e.value)
    t = net.plan_tiled(1, 64, 70000, (64, 4096))
    assert (t["out_h"], t["out_w"]) == (51, 70000 - 13)
    with pytest.raises(fsb.FsError) as e:
        net.plan_tiled(1, 64, 70000, (64, 65535))  # a region of 65548 columns
    assert e.value.status == fsb.FS_ERR_UNSUPPORTED
    with pytest.raises(fsb.FsError) as e:  # the mirrored border extends past the limit
        net.plan(1, 64, 65530, "reflect")
    assert e.value.status == fsb.FS_ERR_UNSUPPORTED
    net.close()


def _wide_layer_net(cin, k):
    layers = [wl.conv(1, 1, cin, "none"), wl.conv(k, cin, 2), wl.fc(1, 2, 2, "softmax")]
    params = [(np.zeros((L["c_out"], L["c_in"], L["k"], L["k"]), np.float32), np.zeros(L["c_out"], np.float32))
              for L in layers]
    return layers, params


@pytest.mark.parametrize("dt,k,cmax", [("f32", 5, 153), ("f32", 3, 245), ("f32", 1, 438),
                                       ("bf16", 5, 265), ("bf16", 3, 450), ("bf16", 1, 862)])
def test_input_channel_limit(dt, k, cmax):
    """A convolution's window holds all its input channels in LDS: the
    largest input channel count a scan takes is planned, one more is refused
    with FS_ERR_UNSUPPORTED (not scanned wrongly), and more than 16384
    channels are refused when the net is created."""
    for cin, fits in ((cmax, True), (cmax + 1, False)):
        layers, params = _wide_layer_net(cin, k)
        w0 = ix.patch_size(layers)
        net = fsb.Net(layers, params, 1, 0, dt, plan_only=True)
        if fits:
            assert net.plan(1, w0 + 40, w0 + 40)["n_launches"] >= 2
        else:
            with pytest.raises(fsb.FsError) as e:
                net.plan(1, w0 + 40, w0 + 40)
            assert e.value.status == fsb.FS_ERR_UNSUPPORTED and "LDS" in str(e.value)
        net.close()
    layers, params = _wide_layer_net(16385, 1)
    with pytest.raises(fsb.FsError) as e:
        fsb.Net(layers, params, 1, 0, dt, plan_only=True)
    assert e.value.status == fsb.FS_ERR_UNSUPPORTED


def test_batch_and_grid_limits():
    """Batch times fragments stays below 2^24 (fragment indices), and a head
    with too many windows is refused instead of overflowing."""
    net = _plan_net(wl.WORKLOADS[2].layers)  # 256 final fragments
    assert net.plan(1000, 95, 95)["out_h"] == 1
    with pytest.raises(fsb.FsError) as e:
        net.plan(65536, 95, 95)
    assert e.value.status == fsb.FS_ERR_UNSUPPORTED and "fragments" in str(e.value)
    with pytest.raises(fsb.FsError) as e:  # 65535 images: a pool's grid passes 2^24 workgroups
        net.plan(65535, 95, 95)
    assert e.value.status == fsb.FS_ERR_UNSUPPORTED and "grid" in str(e.value)
    net.close()
    # a lone 1 x 1 fully connected layer on a 65535 x 65535 image: 2^32 windows
    net = _plan_net([wl.fc(1, 1, 2, "softmax")])
    with pytest.raises(fsb.FsError) as e:
        net.plan(1, 65535, 65535)
    assert e.value.status == fsb.FS_ERR_UNSUPPORTED
    net.close()


def test_binding_tensor_checks():
    """The binding refuses, before any pointer reaches the library, images
    with the wrong channel count, dtype or layout and outputs or workspaces
    that do not match (on the CPU here; the device checks use meta tensors)."""
    torch = pytest.importorskip("torch")
    img = torch.zeros((2, 20, 21, 3))
    shape = (2, 7, 8, 4)
    fsb.check_tensors(img, torch.zeros(shape), torch.zeros(64, dtype=torch.uint8), 3, shape, require_cuda=False)
    bad = [
        (img, None, None, 1),                                   # channels
        (img.double(), None, None, 3),                          # dtype
        (img.permute(0, 2, 1, 3), None, None, 3),               # layout
        (img[0], None, None, 3),                                # rank
        (img, torch.zeros((2, 7, 8, 3)), None, 3),              # output shape
        (img, torch.zeros(shape, dtype=torch.float64), None, 3),
        (img, torch.zeros((2, 8, 7, 4)).transpose(1, 2), None, 3),
        (img, torch.zeros(shape, device="meta"), None, 3),      # output device
        (img, None, torch.zeros((8, 8), dtype=torch.uint8).t(), 3),
        (img, None, torch.zeros(64, dtype=torch.uint8, device="meta"), 3),
    ]
    for im, out, ws, c in bad:
        with pytest.raises(ValueError):
            fsb.check_tensors(im, out, ws, c, shape, require_cuda=False)
    with pytest.raises(ValueError):
        fsb.check_tensors(img, None, None, 3, shape)  # a CPU image for a scan


def test_bench_oracle_window_sample():
    """bench.py's per-patch sample: every image's four corners, the first
    and last window of every final fragment of every image (found by the
    oracle's corner tracking), and 4096 seeded random windows, each once."""
    import sys
    sys.path.insert(0, ROOT)
    import bench
    w = wl.WORKLOADS[4]
    pts = bench.oracle_windows(w)
    assert len(pts) == len(np.unique(pts, axis=0))
    assert pts.min(0).tolist() == [0, 0, 0] and pts.max(0).tolist() == [7, 929, 929]
    fr = ix.reassembly_index(w.layers, w.height, w.width)
    for b in range(w.batch):
        mine = pts[pts[:, 0] == b]
        for Y in (0, 929):
            for X in (0, 929):
                assert ((mine[:, 1] == Y) & (mine[:, 2] == X)).any()
        f = fr[mine[:, 1], mine[:, 2], 0]
        assert set(f.tolist()) == set(range(256))  # every final fragment is hit
    assert 2 * 256 * 8 <= len(pts) <= 2 * 256 * 8 + 32 + 4096


def test_noalloc_scan_limits_without_device():
    """fs_scan_noalloc checks its arguments and the scratch size before any
    device work: a scan whose workspace exceeds the per-GPU scratch array is
    refused with FS_ERR_WORKSPACE (checked with a planning-only net and
    addresses that are never touched)."""
    lib = fsb.load()
    net = _plan_net(wl.WORKLOADS[2].layers)
    scratch = 128 << 20
    assert net.plan(1, 512, 512)["workspace_bytes"] <= scratch < net.plan(1, 1024, 1024)["workspace_bytes"]
    img, out = ctypes.c_void_p(1 << 20), ctypes.c_void_p(2 << 20)
    st = lib.fs_scan_noalloc(net._h, img, 1, 1024, 1024, out, None)
    assert st == fsb.FS_ERR_WORKSPACE and b"fs_scan_noalloc" in lib.fs_last_error()
    st = lib.fs_scan_noalloc(net._h, ctypes.c_void_p((1 << 20) + 4), 1, 512, 512, out, None)
    assert st == fsb.FS_ERR_INVALID_ARG
    st = lib.fs_scan_noalloc(net._h, img, 1, 90, 512, out, None)
    assert st == fsb.FS_ERR_SHAPE
    # within the limit, a planning-only net still never launches
    st = lib.fs_scan_noalloc(net._h, img, 1, 512, 512, out, None)
    assert st == fsb.FS_ERR_INVALID_ARG and b"planning only" in lib.fs_last_error()
    net.close()


def test_plan_cache(monkeypatch):
    """Plans are cached per net and size: a repeated plan is the same, a
    planner switch set in between gives the plan made under it, and planning
    from several threads at once (more sizes than the cache holds) gives
    every thread the single-threaded answers."""
    import threading
    monkeypatch.delenv("FRAGSCAN_POOL_FUSE", raising=False)
    w = wl.WORKLOADS[2]
    net = _plan_net(w.layers)
    a = net.launches(1, 300, 280)
    assert net.launches(1, 300, 280) == a
    monkeypatch.setenv("FRAGSCAN_POOL_FUSE", "0")
    b = net.launches(1, 300, 280)
    assert [L["name"] for L in b] != [L["name"] for L in a] and len(b) == len(a) + 1
    monkeypatch.delenv("FRAGSCAN_POOL_FUSE")
    assert net.launches(1, 300, 280) == a
    sizes = [(1 + i % 3, 95 + 7 * i, 120 + 5 * i) for i in range(24)]
    want = {s: net.plan(*s) for s in sizes}
    errors = []

    def worker(k):
        try:
            for rep in range(20):
                for s in sizes[k % 5:] + sizes[:k % 5]:
                    if net.plan(*s) != want[s]:
                        errors.append(s)
        except Exception as e:  # noqa: BLE001
            errors.append(e)

    th = [threading.Thread(target=worker, args=(k,)) for k in range(6)]
    for t in th:
        t.start()
    for t in th:
        t.join()
    assert not errors, errors[:3]
    net.close()



@pytest.mark.parametrize("seed", range(25))
def test_tables_random_stride_nets(seed):
    """Pools whose stride differs from their size (overlapping or gapped):
    the library's sizes, fragment table and reassembly index agree with the
    oracle's corner tracking bit for bit."""
    rng = np.random.default_rng(4800 + seed)
    layers, (h0, w0), c0 = wl.random_stride_net(rng)
    H = h0 + int(rng.integers(0, 25))
    W = w0 + int(rng.integers(0, 25))
    _check_tables(layers, H, W, c0)


def test_stride_rules():
    """Strides: a pool with stride 0 is the paper's pool; a column stride of
    0 follows the row stride; a stride that does not tile the map, a negative
    stride and a strided convolution are refused."""
    base = [wl.conv(2, 1, 2), wl.pool(3, 2, stride=2), wl.fc(2, 2, 2, "softmax")]
    assert ix.patch_size(base) == 6  # fc 2 -> pool (2-1)*2+3 = 5 -> conv 6
    net = _plan_net(base)
    assert (net.patch, net.info["stride"], net.info["n_fragments"]) == (6, 2, 4)
    net.close()
    only_rows = [dict(L) for L in base]
    del only_rows[1]["stride_x"]  # stride_x follows stride
    net = _plan_net(only_rows)
    assert (net.patch, net.patch_x, net.info["stride_x"]) == (6, 6, 2)
    net.close()
    # stride 3 on a 3x3 pool is the plain pool
    plain = _plan_net([wl.conv(2, 1, 2), wl.pool(3, 2), wl.fc(2, 2, 2, "softmax")])
    same = _plan_net([wl.conv(2, 1, 2), wl.pool(3, 2, stride=3), wl.fc(2, 2, 2, "softmax")])
    assert plain.launches(1, 40, 37) == same.launches(1, 40, 37)
    assert np.array_equal(plain.reassembly_index(40, 37), same.reassembly_index(40, 37))
    plain.close()
    same.close()
    # patch 7: the 6 x 6 map after the conv does not end a stride-2 3x3 window
    params = wl.make_weights(base, 0, 0.1)
    assert _status(base, params, patch=7) == fsb.FS_ERR_SHAPE
    bad = [dict(L) for L in base]
    bad[1]["stride"] = -1
    assert _status(bad, params) == fsb.FS_ERR_INVALID_ARG
    bad = [dict(L) for L in base]
    bad[0]["stride"] = 2
    assert _status(bad, params) == fsb.FS_ERR_UNSUPPORTED
    # a strided pool after a convolution is not fused into it
    layers = [wl.conv(3, 3, 32), wl.pool(3, 32, stride=2), wl.conv(2, 32, 16), wl.pool(2, 16),
              wl.fc(2, 16, 8), wl.fc(1, 8, 2, "softmax")]
    net = _plan_net(layers, c0=3)
    names = [L["name"] for L in net.launches(1, 120, 111)]
    net.close()
    assert not names[0].endswith("+pool") and names[1].startswith("pool_frag<"), names


