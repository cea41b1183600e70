"""The bounds-checked library (libfragscan_debug.so) on the GPU.

Its kernels check every fragment read and write against the true size of the
fragment (the planner's per-axis tables, or Eqs. 6-7 for a pool's children)
and every output-map write against the map.  A scan whose checks all pass
gives the release library's output bit for bit (the checks change no
arithmetic); a failed check comes back as FS_ERR_BOUNDS naming its site.
Failures are forced from the host (FRAGSCAN_DEBUG_SHRINK: one launch's checks
take true sizes one smaller than the real ones), so that every access stays
inside its buffer and every kernel ends normally.
"""
import numpy as np
import pytest

import oracle
from oracle import index as ix
from paper_1302_1700_amd import workloads as wl

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

TOL = {"f32": 1e-4, "bf16": 2e-2}


@pytest.fixture(scope="module")
def fsb():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_1302_1700_amd import fragscan
    fragscan.load()
    fragscan.load(debug=True)
    return fragscan


def _run(fsb, layers, params, img, c0, dt, debug, how="scan", arg=None):
    net = fsb.Net(layers, params, c0, 0, dt, debug=debug)
    x = torch.from_numpy(np.ascontiguousarray(img, np.float32)).cuda()
    try:
        if how == "scan":
            out = net.scan(x)
        elif how == "border":
            out = net.scan(x, border=arg)
        elif how == "tiled":
            out = net.scan_tiled(x, arg)
        else:
            B, H, W, _ = img.shape
            p = net.plan(B, H, W)
            out = torch.empty((B, p["out_h"], p["out_w"], net.n_classes), dtype=torch.float32, device=x.device)
            if how == "noalloc":
                net.scan_noalloc(x, out)
            else:
                net.profile(x, reps=2, out=out)
        torch.cuda.synchronize()
        return out.cpu().numpy()
    finally:
        net.close()


def _same(fsb, layers, params, img, c0, dt="f32", how="scan", arg=None):
    """Debug and release scans agree bit for bit; returns the map."""
    print("debug library", how, arg, dt, img.shape, flush=True)
    rel = _run(fsb, layers, params, img, c0, dt, False, how, arg)
    dbg = _run(fsb, layers, params, img, c0, dt, True, how, arg)
    assert np.array_equal(rel, dbg), how
    return dbg


@pytest.mark.parametrize("wid,B,H,W", [(1, 1, 64, 64), (2, 1, 150, 141), (3, 1, 170, 163), (4, 3, 120, 131),
                                       (5, 1, 140, 151)])
def test_workload_nets(fsb, wid, B, H, W):
    """The five workload nets on small images (gather and vector paths, the
    vector-ALU first layer, fused pools, the fused head, bf16)."""
    w = wl.WORKLOADS[wid]
    params, img = wl.workload_inputs(wid, batch=B, height=H, width=W)
    got = _same(fsb, w.layers, params, img, w.channels, w.dtype)
    ref = oracle.frag_cpu.frag_scan(w.layers, params, img, w.patch)
    assert np.abs(got - ref).max() <= TOL[w.dtype]


@pytest.mark.parametrize("wid", [2, 3, 4, 5])
def test_workload_nets_full_size(fsb, wid):
    """The benchmarked configurations at their full sizes (the grids of many
    rounds, the batch offsets and the tiles the planner picks only there):
    every check passes and the map is the release library's bit for bit."""
    w = wl.WORKLOADS[wid]
    params, img = wl.workload_inputs(wid)
    _same(fsb, w.layers, params, img, w.channels, w.dtype)


@pytest.mark.parametrize("seed", range(4))
def test_random_nets(fsb, seed):
    rng = np.random.default_rng(7000 + seed)
    layers, w0, c0 = wl.random_net(rng, max_c=40)
    params = wl.make_weights(layers, seed, 0.3)
    dt = "bf16" if seed % 2 else "f32"
    img = wl.make_image(seed, 2, w0 + int(rng.integers(0, 40)), w0 + int(rng.integers(0, 40)), c0)
    got = _same(fsb, layers, params, img, c0, dt)
    ref = oracle.patch_forward(layers, params, img, w0)
    assert np.abs(got - ref).max() <= TOL[dt]


@pytest.mark.parametrize("env", [{"FRAGSCAN_POOL_FUSE": "0"}, {"FRAGSCAN_NO_FUSED_HEAD": "1"},
                                 {"FRAGSCAN_STORE": "lds", "FRAGSCAN_POOL_FUSE": "0"},
                                 {"FRAGSCAN_RUN": "1"}, {"FRAGSCAN_ROWTILES": "1", "FRAGSCAN_POOL_FUSE": "0"}])
@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_kernel_paths(fsb, monkeypatch, env, dt):
    """Separate pool and head kernels, restaged stores, run tiles (a tile
    continuing into the next fragment) and row tiles, on ragged fragments."""
    for k, v in env.items():
        monkeypatch.setenv(k, v)
    layers = [wl.conv(3, 3, 32), wl.conv(2, 32, 64), wl.pool(2, 64), wl.conv(2, 64, 40),
              wl.conv(1, 40, 18), wl.pool(2, 18), wl.fc(2, 18, 24), wl.fc(1, 24, 7, "softmax")]
    w0 = ix.patch_size(layers)
    params = wl.make_weights(layers, 21, 0.2)
    img = wl.make_image(22, 2, w0 + 90, w0 + 77, 3)
    got = _same(fsb, layers, params, img, 3, dt)
    ref = oracle.patch_forward(layers, params, img, w0)
    assert np.abs(got - ref).max() <= TOL[dt]


@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_rect_and_strided_pools(fsb, dt):
    """Rectangular kernels and pools, and pools whose stride differs from
    their size (the general pool kernel)."""
    nets = [[wl.conv(3, 3, 32, kx=2), wl.pool(2, 32, kx=3), wl.conv(2, 32, 48, kx=3), wl.pool(3, 48, kx=2),
             wl.fc(2, 48, 24), wl.fc(1, 24, 3, "softmax")],
            [wl.conv(3, 3, 32), wl.pool(3, 32, stride=2), wl.conv(2, 32, 48), wl.pool(2, 48, stride=3),
             wl.fc(2, 48, 24), wl.fc(1, 24, 3, "softmax")]]
    for n, layers in enumerate(nets):
        h0, w0 = ix.patch_hw(layers)
        params = wl.make_weights(layers, 40 + n, 0.2)
        img = wl.make_image(50 + n, 2, h0 + 53, w0 + 61, 3)
        got = _same(fsb, layers, params, img, 3, dt)
        ref = oracle.frag_cpu.frag_scan(layers, params, img, (h0, w0))
        assert np.abs(got - ref).max() <= TOL[dt], n


@pytest.mark.parametrize("how,arg", [("border", "reflect"), ("border", "symmetric"), ("tiled", (37, 29)),
                                     ("noalloc", None), ("profile", None)])
def test_entry_points(fsb, how, arg):
    """Mirrored borders (the mirror pad), the tiled scan, the no-allocation
    entry point and the profiled scan."""
    w = wl.WORKLOADS[2]
    params, img = wl.workload_inputs(2, height=150, width=141)
    _same(fsb, w.layers, params, img, 1, "f32", how, arg)


def _expected_sites(name):
    """Check sites a launch with true sizes one too small must report."""
    if name.startswith("pool_frag"):
        return ["pool parent"]
    if name.startswith("head_softmax"):
        return ["head fragment"]
    sites = ["convolution input window"]
    if name.endswith("+pool"):
        sites.append("fused pool child")
    elif name.endswith("+head"):
        sites.append("fused head output map")
    else:
        sites.append("convolution output")
    return sites


@pytest.mark.parametrize("wid,env", [(2, {}), (3, {}), (5, {}), (2, {"FRAGSCAN_NO_FUSED_HEAD": "1",
                                                                     "FRAGSCAN_POOL_FUSE": "0"})])
def test_failed_checks_reported(fsb, monkeypatch, wid, env):
    """Each launch of the scan in turn checks against sizes one row and one
    column short: the scan returns FS_ERR_BOUNDS naming the launch's check
    sites; the next scan, with the true sizes, passes and matches the
    release library.  The release library ignores the switch."""
    for k, v in env.items():
        monkeypatch.setenv(k, v)
    w = wl.WORKLOADS[wid]
    params, img = wl.workload_inputs(wid, height=150, width=141)
    B, H, W, _ = img.shape
    ref = _run(fsb, w.layers, params, img, w.channels, w.dtype, False)
    net = fsb.Net(w.layers, params, w.channels, 0, w.dtype, debug=True)
    names = [L["name"] for L in net.launches(B, H, W)]
    x = torch.from_numpy(np.ascontiguousarray(img, np.float32)).cuda()
    try:
        for i, name in enumerate(names):
            monkeypatch.setenv("FRAGSCAN_DEBUG_SHRINK", str(i))
            print("forced check failure", wid, env, i, name, flush=True)
            with pytest.raises(fsb.FsError) as e:
                net.scan(x)
            assert e.value.status == fsb.FS_ERR_BOUNDS
            for site in _expected_sites(name):
                assert site in str(e.value), (name, str(e.value))
            monkeypatch.delenv("FRAGSCAN_DEBUG_SHRINK")
            out = net.scan(x)
            torch.cuda.synchronize()
            assert np.array_equal(out.cpu().numpy(), ref), name
        monkeypatch.setenv("FRAGSCAN_DEBUG_SHRINK", "pad")
        with pytest.raises(fsb.FsError) as e:
            net.scan(x, border="reflect")
        assert e.value.status == fsb.FS_ERR_BOUNDS and "mirror pad image" in str(e.value)
    finally:
        net.close()
    monkeypatch.setenv("FRAGSCAN_DEBUG_SHRINK", "0")
    assert np.array_equal(_run(fsb, w.layers, params, img, w.channels, w.dtype, False), ref)
