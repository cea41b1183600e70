"""GPU parity: the HIP scan (through the C-ABI) against the CPU oracle.

Tolerances (max abs on the outputs): float32 1e-4, bf16 (fp32 accumulate)
2e-2, both against the float64 oracle on the float32 weights and image.
Index work (which window lands where) is checked bit-exactly with
position-encoding nets whose arithmetic is exact in both precisions.
"""
import os

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
    """The binding; with FRAGSCAN_TEST_DEBUG=1 every net of these tests is
    loaded into the bounds-checked library instead (a failed check then
    raises FsError, so the whole suite doubles as a memory-safety run)."""
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_1302_1700_amd import fragscan
    fragscan.load()
    if os.environ.get("FRAGSCAN_TEST_DEBUG") != "1":
        return fragscan
    fragscan.load(debug=True)

    class Checked:
        def __getattr__(self, name):
            return getattr(fragscan, name)

        @staticmethod
        def Net(*args, **kw):
            kw.setdefault("debug", True)
            return fragscan.Net(*args, **kw)

    return Checked()


def _scan(fsb, layers, params, img, c0, patch=0, dtype="f32", poison=False):
    net = fsb.Net(layers, params, c0, patch, dtype)
    x = torch.from_numpy(np.ascontiguousarray(img, np.float32)).cuda()
    ws = None
    if poison:
        B, H, W, _ = img.shape
        ws = net.workspace(B, H, W, x.device)
        ws.view(torch.uint8).fill_(0xFF)  # all-ones bytes: NaN in f32 and bf16
    out = net.scan(x, workspace=ws)
    torch.cuda.synchronize()
    res = out.cpu().numpy().astype(np.float64)
    net.close()
    return res


def _sample_patches(layers, B, H, W, n_random, seed):
    """Corners, the first and last window of a spread of final fragments, and
    seeded random windows, as (b, Y, X) rows."""
    h0, w0 = ix.patch_hw(layers)
    ny, nx = H - h0 + 1, W - w0 + 1
    pts = set()
    for b in {0, B - 1}:
        for Y in (0, ny - 1):
            for X in (0, nx - 1):
                pts.add((b, Y, X))
    Sy = Sx = 1
    for L in layers:
        if L["kind"] == "pool":
            Sy *= ix.kyx(L)[0]
            Sx *= ix.kyx(L)[1]
    rng = np.random.default_rng(seed)
    for _ in range(8):
        ry, rx = int(rng.integers(0, min(Sy, ny))), int(rng.integers(0, min(Sx, nx)))
        lastY = ry + (ny - 1 - ry) // Sy * Sy
        lastX = rx + (nx - 1 - rx) // Sx * Sx
        pts.add((0, ry, rx))
        pts.add((B - 1, lastY, lastX))
    for _ in range(n_random):
        pts.add((int(rng.integers(0, B)), int(rng.integers(0, ny)), int(rng.integers(0, nx))))
    return np.array(sorted(pts), np.int32)


# ---- small cases against the full per-patch oracle ---------------------------

def test_workload1_full(fsb):
    w = wl.WORKLOADS[1]
    params, img = wl.workload_inputs(1)
    got = _scan(fsb, w.layers, params, img, w.channels, w.patch)
    ref = oracle.patch_forward(w.layers, params, img, w.patch)
    assert got.shape == ref.shape
    assert np.abs(got - ref).max() <= TOL["f32"]


@pytest.mark.parametrize("seed", range(12))
def test_random_nets_f32(fsb, seed):
    rng = np.random.default_rng(7000 + seed)
    layers, w0, c0 = wl.random_net(rng, max_c=20)
    params = wl.make_weights(layers, seed, 0.3)
    B = int(rng.integers(1, 3))
    H = w0 + int(rng.integers(0, 40))
    W = w0 + int(rng.integers(0, 40))
    img = wl.make_image(seed, B, H, W, c0)
    print("random net", seed, [(L["kind"], L["k"], L["c_in"], L["c_out"]) for L in layers], B, H, W, flush=True)
    got = _scan(fsb, layers, params, img, c0)
    ref = oracle.patch_forward(layers, params, img, w0)
    assert np.abs(got - ref).max() <= TOL["f32"]


@pytest.mark.parametrize("seed", range(6))
def test_random_nets_bf16(fsb, seed):
    rng = np.random.default_rng(8000 + seed)
    layers, w0, c0 = wl.random_net(rng, max_c=40)
    params = wl.make_weights(layers, seed, 0.3)
    H = w0 + int(rng.integers(0, 30))
    W = w0 + int(rng.integers(0, 30))
    img = wl.make_image(seed, 1, H, W, c0)
    got = _scan(fsb, layers, params, img, c0, dtype="bf16")
    ref = oracle.patch_forward(layers, params, img, w0)
    assert np.abs(got - ref).max() <= TOL["bf16"]


def test_channel_multiples_vector_path(fsb):
    """Channel counts that take the vector path (multiples of 16 / 32), three
    pools including a 3x3 one, several tiles per fragment and ragged tails."""
    layers = [wl.conv(2, 3, 32), wl.pool(3, 32), wl.conv(3, 32, 48), wl.pool(2, 48),
              wl.conv(2, 48, 64), wl.pool(2, 64), wl.fc(2, 64, 40), wl.fc(1, 40, 3, "softmax")]
    w0 = ix.patch_size(layers)
    params = wl.make_weights(layers, 5, 0.15)
    img = wl.make_image(6, 2, w0 + 45, w0 + 37, 3)
    ref = oracle.patch_forward(layers, params, img, w0)
    for dt in ("f32", "bf16"):
        got = _scan(fsb, layers, params, img, 3, dtype=dt)
        assert np.abs(got - ref).max() <= TOL[dt], dt


@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_wide_channel_staging(fsb, dt):
    """Window staging for many loads per pixel: 70 channels (gather path,
    more than 64 elements per pixel) and 272 channels (vector path: 68
    16-byte loads per pixel in f32, 34 in bf16), with several tiles and
    ragged fragments."""
    layers = [wl.conv(2, 3, 70), wl.conv(2, 70, 272), wl.pool(2, 272), wl.conv(2, 272, 32),
              wl.fc(2, 32, 16), wl.fc(1, 16, 2, "softmax")]
    w0 = ix.patch_size(layers)
    params = wl.make_weights(layers, 41, 0.08)
    img = wl.make_image(42, 1, w0 + 37, w0 + 30, 3)
    got = _scan(fsb, layers, params, img, 3, dtype=dt)
    ref = oracle.patch_forward(layers, params, img, w0)
    assert np.abs(got - ref).max() <= TOL[dt]


# ---- workload nets on smaller images: full map -------------------------------

@pytest.mark.parametrize("wid,H,W,B", [(2, 150, 141, 1), (3, 170, 163, 1), (4, 120, 131, 3), (5, 140, 151, 1)])
def test_workload_net_small_image(fsb, wid, H, W, B):
    w = wl.WORKLOADS[wid]
    params, img = wl.workload_inputs(wid, batch=B, height=H, width=W)
    got = _scan(fsb, w.layers, params, img, w.channels, 0, w.dtype)
    ref = oracle.frag_cpu.frag_scan(w.layers, params, img, w.patch)
    assert got.shape == ref.shape
    assert np.abs(got - ref).max() <= TOL[w.dtype]
    pts = _sample_patches(w.layers, B, H, W, 24, wid)
    ref_p = oracle.patch_forward(w.layers, params, img, w.patch, pts)
    assert np.abs(got[pts[:, 0], pts[:, 1], pts[:, 2]] - ref_p).max() <= TOL[w.dtype]


# ---- full-size workloads (the benchmarked configurations), sampled ----------

def _fragment_windows(layers, B, H, W):
    """(b, Y, X) of the first and the last window of every final fragment of
    every image (the fragments' extreme pixels: where a wrong size, base or
    stride would show first), from the oracle's own corner tracking."""
    f = ix.reassembly_index(layers, H, W)[..., 0].ravel()
    nx = W - ix.patch_hw(layers)[1] + 1
    _, first = np.unique(f, return_index=True)
    _, last_rev = np.unique(f[::-1], return_index=True)
    last = f.size - 1 - last_rev
    flat = np.concatenate([first, last])
    rows = []
    for b in range(B):
        rows.append(np.stack([np.full(flat.size, b), flat // nx, flat % nx], 1))
    return np.concatenate(rows)


def _full_size_windows(layers, B, H, W, n_random, seed):
    """Every image's corners, the first and last window of every final
    fragment of every image, and n_random seeded random windows."""
    h0, w0 = ix.patch_hw(layers)
    ny, nx = H - h0 + 1, W - w0 + 1
    rng = np.random.default_rng(seed)
    corners = np.array([(b, Y, X) for b in range(B) for Y in (0, ny - 1) for X in (0, nx - 1)])
    rand = np.stack([rng.integers(0, B, n_random), rng.integers(0, ny, n_random), rng.integers(0, nx, n_random)], 1)
    pts = np.concatenate([corners, _fragment_windows(layers, B, H, W), rand])
    return np.unique(pts, axis=0).astype(np.int32)


@pytest.mark.parametrize("wid", [2, 3, 4, 5])
def test_workload_full_size_sampled(fsb, wid):
    """The benchmarked configurations at full size, in the launch
    configuration the benchmark times: every final fragment's first and last
    window in every image, the corners, and 4096 seeded random windows
    against the per-patch oracle; the whole map finite and normalised."""
    w = wl.WORKLOADS[wid]
    params, img = wl.workload_inputs(wid)
    pts = _full_size_windows(w.layers, w.batch, w.height, w.width, 4096, 50 + wid)
    print("full-size workload", wid, img.shape, "windows checked:", len(pts), flush=True)
    got = _scan(fsb, w.layers, params, img, w.channels, 0, w.dtype)
    assert got.shape == (w.batch, w.out_h, w.out_w, w.n_classes)
    assert np.isfinite(got).all()
    assert np.abs(got.sum(-1) - 1.0).max() <= 1e-5
    F = ix.n_fragments(w.layers)
    assert len(pts) >= 4096 + min(2 * F, w.out_h * w.out_w) * w.batch // 2
    ref = oracle.patch_forward(w.layers, params, img, w.patch, pts)
    assert np.abs(got[pts[:, 0], pts[:, 1], pts[:, 2]] - ref).max() <= TOL[w.dtype]


def test_workload2_full_map_cpu_fragment(fsb):
    """Net N4 on the full 512 x 512 image: every one of the 174,724 outputs
    against the CPU fragment method (float64), itself pinned to the per-patch
    definition."""
    w = wl.WORKLOADS[2]
    params, img = wl.workload_inputs(2)
    got = _scan(fsb, w.layers, params, img, w.channels, 0, w.dtype)
    ref = oracle.frag_cpu.frag_scan(w.layers, params, img, w.patch)
    assert got.shape == ref.shape == (1, 418, 418, 2)
    assert np.abs(got - ref).max() <= TOL["f32"]


@pytest.mark.parametrize("wid", [3, 4, 5])
def test_workload_full_map_dilated(fsb, wid):
    """Full-size benchmarked configurations, every output of the map against
    the whole-image formulation with dilated library convolutions and
    max-pools (float64, torch CPU; pinned to the per-patch definition by the
    oracle tests): workloads 3 and 5 whole, workload 4's first and last image
    of its batch of eight (~8 s of CPU per 1024^2 image)."""
    from helpers import dilated_scan
    w = wl.WORKLOADS[wid]
    params, img = wl.workload_inputs(wid)
    got = _scan(fsb, w.layers, params, img, w.channels, 0, w.dtype)
    for b in sorted({0, w.batch - 1}):
        print("full map vs dilated formulation", wid, "image", b, flush=True)
        ref = dilated_scan(w.layers, params, img[b:b + 1])
        assert got[b:b + 1].shape == ref.shape
        assert np.abs(got[b:b + 1] - ref).max() <= TOL[w.dtype], b


@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_image_side_limit(fsb, dt):
    """Images whose width or height is 65,535, the largest side a scan takes
    (fragment sizes travel in 16-bit tables): the tiny workload net (small-K
    first layer) and a matrix-core net, the whole map against the dilated
    whole-image formulation and sampled windows against the per-patch
    oracle."""
    from helpers import dilated_scan
    nets = [(wl.WORKLOADS[1].layers, 1),
            ([wl.conv(2, 3, 32), wl.pool(2, 32), wl.conv(2, 32, 32), wl.pool(2, 32), wl.fc(2, 32, 16),
              wl.fc(1, 16, 2, "softmax")], 3)]
    for n, (layers, c0) in enumerate(nets):
        w0 = ix.patch_size(layers)
        params = wl.make_weights(layers, 120 + n, 0.3)
        for H, W in ((w0 + 5, 65535), (65535, w0 + 3)):
            img = wl.make_image(130 + n, 1, H, W, c0)
            print("side limit", dt, n, (H, W), flush=True)
            got = _scan(fsb, layers, params, img, c0, dtype=dt)
            ref = dilated_scan(layers, params, img)
            assert got.shape == ref.shape == (1, H - w0 + 1, W - w0 + 1, 2)
            assert np.abs(got - ref).max() <= TOL[dt], (n, H, W)
            pts = _sample_patches(layers, 1, H, W, 64, 140 + n)
            ref_p = oracle.patch_forward(layers, params, img, w0, pts)
            assert np.abs(got[pts[:, 0], pts[:, 1], pts[:, 2]] - ref_p).max() <= TOL[dt], (n, H, W)


def test_workload3_logits(fsb):
    """Workload 3's probabilities sit within 1e-3 of 1/2, so also compare the
    logits (last layer without softmax) on a relative scale."""
    w = wl.WORKLOADS[3]
    layers = [dict(L) for L in w.layers]
    layers[-1]["act"] = "none"
    params, img = wl.workload_inputs(3, height=400, width=380)
    got = _scan(fsb, layers, params, img, 3)
    pts = _sample_patches(layers, 1, 400, 380, 300, 3)
    ref = oracle.patch_forward(layers, params, img, w.patch, pts)
    g = got[pts[:, 0], pts[:, 1], pts[:, 2]]
    spread = np.abs(ref).max()
    assert np.abs(g - ref).max() <= 1e-4 * spread
    # a one-pixel shift of the output map would be far outside the bound
    shifted = got[pts[:, 0], pts[:, 1], np.minimum(pts[:, 2] + 1, got.shape[2] - 1)]
    assert np.abs(shifted - ref).max() > 20 * np.abs(g - ref).max()


# ---- exact index checks -----------------------------------------------------

def _probe_net(pools, ks, c):
    """Convolutions that copy one channel through a single tap and max-pools
    of the given sizes: on an image whose values grow along y and x, every
    max is the window's last pixel, so the output is the image value at a
    fixed offset from the window's corner, exactly."""
    layers, params = [], []
    for kind, k in zip(pools, ks):
        if kind == "pool":
            layers.append(wl.pool(k, c))
            params.append(None)
        else:
            layers.append(wl.conv(k, c, c, "none"))
            wt = np.zeros((c, c, k, k), np.float32)
            for i in range(c):
                wt[i, i, k - 1, 0] = 1.0  # bottom-left tap
            params.append((wt, np.zeros(c, np.float32)))
    w_L = 2
    layers.append(wl.fc(w_L, c, c, "none"))
    wt = np.zeros((c, c, w_L, w_L), np.float32)
    for i in range(c):
        wt[i, i, 0, 1] = 1.0
    params.append((wt, np.zeros(c, np.float32)))
    return layers, params


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_reassembly_bit_exact(fsb, dtype):
    kinds = ["conv", "pool", "conv", "pool", "conv", "pool"]
    ks = [3, 2, 2, 3, 2, 2]
    layers, params = _probe_net(kinds, ks, 3)
    w0 = ix.patch_size(layers)
    B, H, W = 2, w0 + 83, w0 + 71
    yy, xx = np.meshgrid(np.arange(H), np.arange(W), indexing="ij")
    img = np.zeros((B, H, W, 3), np.float32)
    for b in range(B):
        # every value is an integer below 256, exact in bf16
        img[b, :, :, 0] = yy % 128 + 64 * b
        img[b, :, :, 1] = xx % 128
        img[b, :, :, 2] = (yy // 128) * 16 + xx // 128 + 128 * b
    got = _scan(fsb, layers, params, img, 3, dtype=dtype)
    ref = oracle.patch_forward(layers, params, img, w0)
    assert np.array_equal(got, ref)


def test_index_probe_table_agrees(fsb):
    """The host reassembly index of the library and the oracle agree, and the
    probe output decodes to each window's own corner."""
    layers, params = _probe_net(["pool", "conv", "pool"], [2, 2, 3], 2)
    w0 = ix.patch_size(layers)
    H, W = w0 + 50, w0 + 61
    yy, xx = np.meshgrid(np.arange(H), np.arange(W), indexing="ij")
    img = np.stack([yy, xx], -1)[None].astype(np.float32)
    got = _scan(fsb, layers, params, img, 2)
    ny, nx = H - w0 + 1, W - w0 + 1
    Y, X = np.meshgrid(np.arange(ny), np.arange(nx), indexing="ij")
    off_y = got[0, :, :, 0] - Y
    off_x = got[0, :, :, 1] - X
    assert (off_y == off_y[0, 0]).all() and (off_x == off_x[0, 0]).all()
    net = fsb.Net(layers, params, 2)
    assert np.array_equal(net.reassembly_index(H, W), ix.reassembly_index(layers, H, W).astype(np.int32))
    net.close()


# ---- edge cases ---------------------------------------------------------------

@pytest.mark.parametrize("extra", [0, 1, 3, 9])
def test_small_images_empty_fragments(fsb, extra):
    """H = w_0 + extra with extra below the pooling stride: most final
    fragments are empty."""
    w = wl.WORKLOADS[2]
    params, img = wl.workload_inputs(2, height=95 + extra, width=95 + 2 * extra)
    got = _scan(fsb, w.layers, params, img, 1)
    ref = oracle.patch_forward(w.layers, params, img, 95)
    assert np.abs(got - ref).max() <= TOL["f32"]


def test_poisoned_workspace(fsb):
    """Fill the workspace with NaN bytes first: a read of padding or of
    anything not written in this scan would show up in the outputs."""
    w = wl.WORKLOADS[5]
    params, img = wl.workload_inputs(5, height=133, width=127)
    ref = oracle.frag_cpu.frag_scan(w.layers, params, img, w.patch)
    for dt in ("f32", "bf16"):
        got = _scan(fsb, w.layers, params, img, 3, 0, dt, poison=True)
        assert np.isfinite(got).all()
        assert np.abs(got - ref).max() <= TOL[dt]


def test_repeat_is_deterministic(fsb):
    w = wl.WORKLOADS[2]
    params, img = wl.workload_inputs(2, height=200, width=180)
    net = fsb.Net(w.layers, params, 1)
    x = torch.from_numpy(img).cuda()
    a = net.scan(x).clone()
    b = net.scan(x).clone()
    torch.cuda.synchronize()
    assert torch.equal(a, b)
    # the profiled scan repeats every launch back to back; its output is the
    # plain scan's
    c = torch.full_like(a, float("nan"))
    ms = net.profile(x, reps=3, out=c)
    torch.cuda.synchronize()
    assert len(ms) == len(net.launches(1, 200, 180)) and all(m > 0 for m in ms)
    assert torch.equal(a, c)
    net.close()


def test_unfused_head_paths(fsb, monkeypatch):
    """The separate head kernel (last layer not folded into the convolution
    before it): forced off by the environment switch, and by a last layer with
    more classes than the fused epilogue takes."""
    w = wl.WORKLOADS[2]
    params, img = wl.workload_inputs(2, height=140, width=150)
    ref = oracle.frag_cpu.frag_scan(w.layers, params, img, w.patch)
    monkeypatch.setenv("FRAGSCAN_NO_FUSED_HEAD", "1")
    got = _scan(fsb, w.layers, params, img, 1)
    assert np.abs(got - ref).max() <= TOL["f32"]
    monkeypatch.delenv("FRAGSCAN_NO_FUSED_HEAD")
    layers = [wl.conv(3, 2, 16), wl.pool(2, 16), wl.conv(2, 16, 32), wl.pool(2, 32),
              wl.fc(2, 32, 24), wl.fc(1, 24, 7, "softmax")]
    w0 = ix.patch_size(layers)
    params = wl.make_weights(layers, 3, 0.3)
    img = wl.make_image(4, 2, w0 + 29, w0 + 33, 2)
    ref = oracle.patch_forward(layers, params, img, w0)
    for dt in ("f32", "bf16"):
        got = _scan(fsb, layers, params, img, 2, dtype=dt)
        assert np.abs(got - ref).max() <= TOL[dt], dt


@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_head_sibling_order(fsb, monkeypatch, dt):
    """Fused-head tiles numbered with the fragment column fastest (the x
    siblings, whose outputs interleave in the map's columns, side by side) or
    in fragment order: the same map bit for bit, and the oracle's values.
    The rectangular net (2 x 3 and 3 x 2 pools: 6 x 6 final fragments) on
    ragged fragments, two images; N4 (16 x 16 final fragments) with the FC
    tile the planner picks (bf16 N4 runs the separate head kernel)."""
    cases = [(_rect_mfma_net(), 65, (2, 16 + 97, 25 + 131, 3), (16, 25), 3)]
    w = wl.WORKLOADS[2]
    cases.append((w.layers, 67, (1, w.patch + 83, w.patch + 121, 1), w.patch, 1))
    for layers, seed, shape, patch, c0 in cases:
        params = wl.make_weights(layers, seed, 0.15)
        img = wl.make_image(seed + 1, *shape)
        got = {}
        for xs in ("1", "0"):
            monkeypatch.setenv("FRAGSCAN_XSIB", xs)
            print("head sibling order", dt, shape, xs, flush=True)
            got[xs] = _scan(fsb, layers, params, img, c0, 0, dt)
        assert np.array_equal(got["1"], got["0"])
        ref = oracle.frag_cpu.frag_scan(layers, params, img, patch)
        assert np.abs(got["1"] - ref).max() <= TOL[dt]


def test_padding_block_and_half_swap(fsb, monkeypatch):
    """N4's FC1 (200 outputs in 14 channel blocks) on the 7 x 2 register tile:
    the wave whose half ends in the padding block skips that block's
    products, and (head fused) alternate workgroups swap the halves between
    the two wave columns.  With the swap and without it the map is the same
    bit for bit, fused head or not, and the oracle's."""
    w = wl.WORKLOADS[2]
    H, W = w.patch + 83, w.patch + 121
    params, img = wl.workload_inputs(2, batch=2, height=H, width=W)
    ref = oracle.frag_cpu.frag_scan(w.layers, params, img, w.patch)
    monkeypatch.setenv("FRAGSCAN_WIDE", "0")
    for fused in ("1", "0"):
        if fused == "0":
            monkeypatch.setenv("FRAGSCAN_NO_FUSED_HEAD", "1")
        got = {}
        for sw in ("1", "0"):
            monkeypatch.setenv("FRAGSCAN_SWAP", sw)
            net = fsb.Net(w.layers, params, 1, 0, "f32")
            names = [L["name"] for L in net.launches(2, H, W)]
            net.close()
            print("padding skip / half swap", fused, sw, names, flush=True)
            assert any(n.startswith("conv_frag_mfma<4, 7, 2, 1,") for n in names), names
            got[sw] = _scan(fsb, w.layers, params, img, 1)
        assert np.array_equal(got["1"], got["0"]), fused
        assert np.abs(got["1"] - ref).max() <= TOL["f32"], fused


@pytest.mark.parametrize("tile", ["2:4,3,1,16,2;4:8,3,1,16,4;6:4,3,1,0,2;8:4,7,2,0,2",
                                  "2:8,3,1,0,4;4:4,3,1,0,2;8:2,13,1,0,2"])
def test_split_k_tiles(fsb, monkeypatch, tile):
    """Register tiles whose waves split the K steps (partial sums reduced
    through LDS), forced through the tile override on net N4."""
    w = wl.WORKLOADS[2]
    params, img = wl.workload_inputs(2, height=171, width=160)
    ref = oracle.frag_cpu.frag_scan(w.layers, params, img, w.patch)
    monkeypatch.setenv("FRAGSCAN_TILE", tile)
    got = _scan(fsb, w.layers, params, img, 1)
    assert np.abs(got - ref).max() <= TOL["f32"]


def _scan_border(fsb, layers, params, img, c0, mode, dtype="f32"):
    net = fsb.Net(layers, params, c0, 0, dtype)
    x = torch.from_numpy(np.ascontiguousarray(img, np.float32)).cuda()
    out = net.scan(x, border=mode)
    torch.cuda.synchronize()
    res = out.cpu().numpy().astype(np.float64)
    net.close()
    return res


@pytest.mark.parametrize("mode", ["reflect", "symmetric"])
def test_mirrored_borders_full(fsb, mode):
    """Section 3.2's mirrored edges: H x W outputs, each the window centred on
    its pixel; workload 1's net (even w_0 = 14: 6 rows / columns before, 7
    after), B = 2, full map against the per-patch oracle on the extended
    image."""
    w = wl.WORKLOADS[1]
    params, _ = wl.workload_inputs(1)
    img = wl.make_image(41, 2, 40, 37, 1)
    ref = oracle.border.scan_mirrored(w.layers, params, img, w.patch, mode)
    got = _scan_border(fsb, w.layers, params, img, 1, mode)
    assert got.shape == ref.shape == (2, 40, 37, 2)
    assert np.abs(got - ref).max() <= TOL["f32"]


@pytest.mark.parametrize("mode", ["reflect", "symmetric"])
def test_mirrored_image_smaller_than_border(fsb, mode):
    """A 3 x 2 image under a 14 x 14 window: the border is mirrored
    repeatedly; single-pixel rows use the one pixel."""
    w = wl.WORKLOADS[1]
    params, _ = wl.workload_inputs(1)
    for H, W in ((3, 2), (1, 5)):
        img = wl.make_image(42, 1, H, W, 1)
        ref = oracle.border.scan_mirrored(w.layers, params, img, w.patch, mode)
        got = _scan_border(fsb, w.layers, params, img, 1, mode)
        assert np.abs(got - ref).max() <= TOL["f32"], (H, W)


def test_mirrored_n4_sampled(fsb):
    """Net N4 (odd w_0 = 95, 47 pixels each side) on a 60 x 70 image, smaller
    than the window: sampled windows, corners included."""
    w = wl.WORKLOADS[2]
    params, _ = wl.workload_inputs(2)
    img = wl.make_image(43, 1, 60, 70, 1)
    got = _scan_border(fsb, w.layers, params, img, 1, "reflect")
    rng = np.random.default_rng(44)
    pts = {(0, 0, 0), (0, 59, 69), (0, 0, 69), (0, 59, 0)}
    for _ in range(60):
        pts.add((0, int(rng.integers(0, 60)), int(rng.integers(0, 70))))
    pts = np.array(sorted(pts), np.int32)
    ref = oracle.border.scan_mirrored(w.layers, params, img, w.patch, "reflect", pts)
    assert np.abs(got[pts[:, 0], pts[:, 1], pts[:, 2]] - ref).max() <= TOL["f32"]


def test_mirrored_bf16(fsb):
    w = wl.WORKLOADS[5]
    params, _ = wl.workload_inputs(5, height=61, width=61)
    img = wl.make_image(45, 1, 50, 47, 3)
    got = _scan_border(fsb, w.layers, params, img, 3, "symmetric", "bf16")
    rng = np.random.default_rng(46)
    pts = np.array(sorted({(0, int(rng.integers(0, 50)), int(rng.integers(0, 47))) for _ in range(60)}
                          | {(0, 0, 0), (0, 49, 46)}), np.int32)
    ref = oracle.border.scan_mirrored(w.layers, params, img, w.patch, "symmetric", pts)
    assert np.abs(got[pts[:, 0], pts[:, 1], pts[:, 2]] - ref).max() <= TOL["bf16"]


@pytest.mark.parametrize("fuse", ["0", "1"])
@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_pool_fusion_modes(fsb, monkeypatch, fuse, dt):
    """Convolutions with the following max-pool fused into their epilogue (or
    not): 2x2 and 3x3 pools, channel counts on and off the 16-byte grid
    (vector and per-channel maxima), the gather and the vector path, ragged
    fragments, B = 2."""
    layers = [wl.conv(2, 3, 32), wl.pool(3, 32), wl.conv(2, 32, 18), wl.pool(2, 18),
              wl.conv(2, 18, 64), wl.pool(2, 64), wl.fc(2, 64, 24), wl.fc(1, 24, 3, "softmax")]
    w0 = ix.patch_size(layers)
    params = wl.make_weights(layers, 21, 0.2)
    img = wl.make_image(22, 2, w0 + 37, w0 + 44, 3)
    ref = oracle.patch_forward(layers, params, img, w0)
    monkeypatch.setenv("FRAGSCAN_POOL_FUSE", fuse)
    net = fsb.Net(layers, params, 3, 0, dt)
    names = [L["name"] for L in net.launches(2, w0 + 37, w0 + 44)]
    net.close()
    assert sum(n.endswith("+pool") for n in names) == (3 if fuse == "1" else 0), names
    got = _scan(fsb, layers, params, img, 3, dtype=dt)
    assert np.abs(got - ref).max() <= TOL[dt]


@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_pool_fusion_bit_exact(fsb, monkeypatch, dt):
    """A pool fused into the convolution's epilogue gives the values of the
    separate pool kernel bit for bit (same K walk per pixel, and the maximum
    is exact): 3x3 and 2x2 pools, 32 and 64 channels (one wave per pixel
    block, no split K), ragged fragments, B = 2."""
    layers = [wl.conv(2, 3, 32), wl.pool(3, 32), wl.conv(3, 32, 32), wl.pool(2, 32),
              wl.conv(2, 32, 64), wl.pool(2, 64), wl.fc(2, 64, 24), wl.fc(1, 24, 3, "softmax")]
    w0 = ix.patch_size(layers)
    params = wl.make_weights(layers, 71, 0.2)
    img = wl.make_image(72, 2, w0 + 53, w0 + 61, 3)
    outs = {}
    for fuse in ("0", "1"):
        monkeypatch.setenv("FRAGSCAN_POOL_FUSE", fuse)
        net = fsb.Net(layers, params, 3, 0, dt)
        names = [L["name"] for L in net.launches(2, img.shape[1], img.shape[2])]
        net.close()
        assert sum(n.endswith("+pool") for n in names) == (3 if fuse == "1" else 0), names
        print("pool fusion bit-exact", dt, fuse, names, flush=True)
        outs[fuse] = _scan(fsb, layers, params, img, 3, dtype=dt)
    assert np.array_equal(outs["0"], outs["1"])
    pts = np.array([(b, y, x) for b in range(2) for y in (0, 17, img.shape[1] - w0)
                    for x in (0, 29, img.shape[2] - w0)], np.int32)
    ref = oracle.patch_forward(layers, params, img, w0, pts)
    assert np.abs(outs["1"][pts[:, 0], pts[:, 1], pts[:, 2]] - ref).max() <= TOL[dt]


def test_pool_fusion_split_k(fsb, monkeypatch):
    """Split-K (two waves per pixel block) feeding the fused pool."""
    layers = [wl.conv(2, 1, 48), wl.pool(2, 48), wl.conv(3, 48, 48), wl.pool(2, 48),
              wl.fc(2, 48, 20), wl.fc(1, 20, 2, "softmax")]
    w0 = ix.patch_size(layers)
    params = wl.make_weights(layers, 23, 0.1)
    img = wl.make_image(24, 1, w0 + 53, w0 + 40, 1)
    ref = oracle.patch_forward(layers, params, img, w0)
    monkeypatch.setenv("FRAGSCAN_POOL_FUSE", "1")
    monkeypatch.setenv("FRAGSCAN_TILE", "2:4,3,1,0,2")
    got = _scan(fsb, layers, params, img, 1)
    assert np.abs(got - ref).max() <= TOL["f32"]


@pytest.mark.parametrize("store", ["direct", "lds"])
@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_store_modes(fsb, monkeypatch, store, dt):
    """Both epilogue store paths on every layer: channel counts that pair
    bf16 blocks (32, 64), leave them unpaired (40), and are not multiples of
    8 or 4 (18), on the vector and the gather path, several tiles and ragged
    fragment sizes."""
    layers = [wl.conv(3, 3, 32), wl.conv(2, 32, 64), wl.pool(2, 64), wl.conv(2, 64, 40),
              wl.conv(1, 40, 18), wl.pool(2, 18), wl.fc(2, 18, 24), wl.fc(1, 24, 3, "softmax")]
    w0 = ix.patch_size(layers)
    params = wl.make_weights(layers, 11, 0.2)
    img = wl.make_image(12, 2, w0 + 41, w0 + 29, 3)
    ref = oracle.patch_forward(layers, params, img, w0)
    monkeypatch.setenv("FRAGSCAN_STORE", store)
    got = _scan(fsb, layers, params, img, 3, dtype=dt)
    assert np.abs(got - ref).max() <= TOL[dt]


@pytest.mark.parametrize("big", [False, True])
@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_run_tiles(fsb, monkeypatch, dt, big):
    """Run tiles (a tile continues into the next fragment) give the same
    values as one tile sequence per fragment, bit for bit: the split-K vector
    layer on the smaller image, the gather layer with the fused head on the
    larger (pools not fused there); two images of ragged fragments."""
    layers = [wl.conv(3, 3, 32), wl.conv(2, 32, 64), wl.pool(2, 64), wl.conv(2, 64, 40),
              wl.conv(1, 40, 18), wl.pool(2, 18), wl.fc(2, 18, 24), wl.fc(1, 24, 3, "softmax")]
    w0 = ix.patch_size(layers)
    params = wl.make_weights(layers, 21, 0.2)
    H, W = (w0 + 90, w0 + 77) if big else (w0 + 41, w0 + 29)
    img = wl.make_image(22, 2, H, W, 3)
    monkeypatch.setenv("FRAGSCAN_POOL_FUSE", "0" if big else "")
    monkeypatch.setenv("FRAGSCAN_RUN", "1")
    run = _scan(fsb, layers, params, img, 3, dtype=dt)
    monkeypatch.setenv("FRAGSCAN_RUN", "0")
    per_frag = _scan(fsb, layers, params, img, 3, dtype=dt)
    assert np.array_equal(run, per_frag)
    ref = oracle.patch_forward(layers, params, img, w0)
    assert np.abs(run - ref).max() <= TOL[dt]


@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_row_tiles(fsb, monkeypatch, dt):
    """Tiles of whole band rows (a narrower last band gets fewer pixels per
    tile) give the same values as tiles of mt pixels, bit for bit, on layers
    with several bands and ragged fragments; pools unfused so the plain conv
    tiles run everywhere."""
    layers = [wl.conv(3, 3, 32), wl.conv(2, 32, 48), wl.pool(2, 48), wl.conv(3, 48, 32),
              wl.pool(2, 32), wl.fc(2, 32, 24), wl.fc(1, 24, 3, "softmax")]
    w0 = ix.patch_size(layers)
    params = wl.make_weights(layers, 31, 0.2)
    img = wl.make_image(32, 2, w0 + 141, w0 + 117, 3)
    monkeypatch.setenv("FRAGSCAN_POOL_FUSE", "0")
    monkeypatch.setenv("FRAGSCAN_ROWTILES", "1")
    rows = _scan(fsb, layers, params, img, 3, dtype=dt)
    monkeypatch.setenv("FRAGSCAN_ROWTILES", "0")
    pix = _scan(fsb, layers, params, img, 3, dtype=dt)
    assert np.array_equal(rows, pix)
    ref = oracle.patch_forward(layers, params, img, w0)
    assert np.abs(rows - ref).max() <= TOL[dt]


@pytest.mark.parametrize("wid", [2, 5])
def test_lds_padding(fsb, monkeypatch, wid):
    """The per-pixel LDS padding only moves the window in LDS: without it the
    scan gives the same values bit for bit."""
    w = wl.WORKLOADS[wid]
    params, img = wl.workload_inputs(wid, height=140, width=131)
    padded = _scan(fsb, w.layers, params, img, w.channels, 0, w.dtype)
    monkeypatch.setenv("FRAGSCAN_LDS_PAD", "0")
    packed = _scan(fsb, w.layers, params, img, w.channels, 0, w.dtype)
    assert np.array_equal(padded, packed)


@pytest.mark.parametrize("wid,B,H,W,tiles", [
    (2, 1, 160, 150, [(17, 23), (5, 64), (1, 1000), (1000, 1000)]),
    (4, 2, 130, 121, [(9, 11)]),
    (3, 1, 170, 163, [(31, 7)]),
    (5, 1, 140, 131, [(20, 33), (7, 80)]),
    (1, 1, 64, 64, [(1, 1), (50, 2)]),
])
def test_tiled_scan(fsb, wid, B, H, W, tiles):
    """Output tiles scanned one after another, each over the image region
    its windows cover, give the untiled scan's values bit for bit (ragged
    last tiles, one-row and one-window tiles, a tile larger than the map)."""
    w = wl.WORKLOADS[wid]
    params, img = wl.workload_inputs(wid, batch=B, height=H, width=W)
    net = fsb.Net(w.layers, params, w.channels, 0, w.dtype)
    x = torch.from_numpy(np.ascontiguousarray(img, np.float32)).cuda()
    ref = net.scan(x).cpu().numpy()
    for tile in tiles:
        print("tiled scan", wid, B, H, W, tile, flush=True)
        out = torch.full_like(torch.from_numpy(ref), float("nan")).cuda()
        net.scan_tiled(x, tile, out=out)
        torch.cuda.synchronize()
        assert np.array_equal(out.cpu().numpy(), ref), tile
    net.close()


def _seam_windows(B, ny, nx, th, tw, rng, per_line=6):
    """Windows on both sides of every boundary between output tiles of
    th x tw windows, and at every crossing of two boundaries."""
    pts = set()
    rows = [r for k in range(1, -(-ny // th)) for r in (k * th - 1, k * th)]
    cols = [c for k in range(1, -(-nx // tw)) for c in (k * tw - 1, k * tw)]
    for b in range(B):
        for r in rows:
            for c in rng.integers(0, nx, per_line):
                pts.add((b, r, int(c)))
            for c in cols:
                pts.add((b, r, c))
        for c in cols:
            for r in rng.integers(0, ny, per_line):
                pts.add((b, int(r), c))
        for Y in (0, ny - 1):
            for X in (0, nx - 1):
                pts.add((b, Y, X))
    return np.array(sorted(pts), np.int32)


@pytest.mark.parametrize("wid,B,H,W,tile", [
    (2, 1, 330, 301, (61, 47)),
    (4, 2, 260, 231, (37, 64)),
    (3, 1, 290, 270, (100, 81)),
    (5, 1, 200, 190, (45, 29)),
])
def test_tiled_scan_seams_against_oracle(fsb, wid, B, H, W, tile):
    """The tiled scan against the per-patch oracle on windows next to every
    tile seam (each tile recomputes the image rows and columns it shares with
    its neighbours), every seam crossing and the corners."""
    w = wl.WORKLOADS[wid]
    params, img = wl.workload_inputs(wid, batch=B, height=H, width=W)
    net = fsb.Net(w.layers, params, w.channels, 0, w.dtype)
    x = torch.from_numpy(np.ascontiguousarray(img, np.float32)).cuda()
    out = torch.full((B, H - w.patch + 1, W - w.patch + 1, w.n_classes), float("nan"), device="cuda")
    net.scan_tiled(x, tile, out=out)
    torch.cuda.synchronize()
    got = out.cpu().numpy().astype(np.float64)
    net.close()
    assert np.isfinite(got).all()
    pts = _seam_windows(B, H - w.patch + 1, W - w.patch + 1, tile[0], tile[1], np.random.default_rng(wid))
    print("tiled seams", wid, tile, len(pts), flush=True)
    ref = oracle.patch_forward(w.layers, params, img, w.patch, pts)
    assert np.abs(got[pts[:, 0], pts[:, 1], pts[:, 2]] - ref).max() <= TOL[w.dtype]


@pytest.mark.parametrize("wid,mode", [(1, "0"), (3, "0"), (2, "1"), (5, "1")])
def test_conv_kernel_choice(fsb, monkeypatch, wid, mode):
    """Small-K layers take either the per-pixel vector-ALU kernel or the
    matrix-core gather kernel; force the one the planner does not pick by
    default for the workload's first layers."""
    w = wl.WORKLOADS[wid]
    H = {1: 64, 2: 140, 3: 150, 5: 120}[wid]
    params, img = wl.workload_inputs(wid, height=H, width=H + 9)
    ref = oracle.frag_cpu.frag_scan(w.layers, params, img, w.patch)
    monkeypatch.setenv("FRAGSCAN_DIRECT", mode)
    got = _scan(fsb, w.layers, params, img, w.channels, 0, w.dtype)
    assert np.abs(got - ref).max() <= TOL[w.dtype]


# ---- rectangular kernels, pools and windows (Section 2: per axis) ----------

@pytest.mark.parametrize("seed", range(10))
def test_rect_random_nets(fsb, seed):
    """Random stacks of rectangular kernels and pools, full output map
    against the fragment oracle and sampled windows against the per-patch
    oracle; odd seeds in bf16."""
    rng = np.random.default_rng(7000 + seed)
    layers, (h0, w0), c0 = wl.random_rect_net(rng)
    dt = "bf16" if seed % 2 else "f32"
    B = 1 + seed % 2
    H, W = h0 + int(rng.integers(0, 40)), w0 + int(rng.integers(0, 40))
    params = wl.make_weights(layers, 7100 + seed, 0.4)
    img = wl.make_image(7200 + seed, B, H, W, c0)
    print("rect net", seed, [(L["kind"], ix.kyx(L)) for L in layers], (B, H, W), dt, flush=True)
    got = _scan(fsb, layers, params, img, c0, 0, dt)
    ref = oracle.frag_cpu.frag_scan(layers, params, img, (h0, w0))
    assert got.shape == ref.shape == (B, H - h0 + 1, W - w0 + 1, layers[-1]["c_out"])
    assert np.abs(got - ref).max() <= TOL[dt]
    pts = _sample_patches(layers, B, H, W, 16, seed)
    ref_p = oracle.patch_forward(layers, params, img, (h0, w0), pts)
    assert np.abs(got[pts[:, 0], pts[:, 1], pts[:, 2]] - ref_p).max() <= TOL[dt]


def _rect_mfma_net():
    """Matrix-core channel counts with 3x2 / 2x3 kernels and 2x3 / 3x2 pools:
    a 16 x 25 window, 36 final fragments."""
    layers = [wl.conv(3, 3, 32, kx=2), wl.pool(2, 32, kx=3), wl.conv(2, 32, 48, kx=3), wl.pool(3, 48, kx=2),
              wl.fc(2, 48, 16, kx=3), wl.fc(1, 16, 2, "softmax")]
    assert ix.patch_hw(layers) == (16, 25)
    return layers


@pytest.mark.parametrize("fuse", ["0", "1"])
@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_rect_mfma_net(fsb, monkeypatch, dt, fuse):
    """Vector-path matrix-core layers, pools fused into the convolutions or
    not, the head fused into the last 2 x 3 layer, two images."""
    layers = _rect_mfma_net()
    params = wl.make_weights(layers, 61, 0.15)
    img = wl.make_image(62, 2, 16 + 93, 25 + 118, 3)
    monkeypatch.setenv("FRAGSCAN_POOL_FUSE", fuse)
    net = fsb.Net(layers, params, 3, 0, dt)
    names = [L["name"] for L in net.launches(2, img.shape[1], img.shape[2])]
    net.close()
    assert sum(n.endswith("+pool") or "+pool+" in n for n in names) == (2 if fuse == "1" else 0), names
    print("rect mfma", dt, fuse, names, flush=True)
    got = _scan(fsb, layers, params, img, 3, 0, dt)
    ref = oracle.frag_cpu.frag_scan(layers, params, img, (16, 25))
    assert np.abs(got - ref).max() <= TOL[dt]


@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_rect_tile_variants(fsb, monkeypatch, dt):
    """The same values, bit for bit, from the gather path for the first
    layer, from run tiles, and from row tiles, on the rectangular net."""
    layers = _rect_mfma_net()
    params = wl.make_weights(layers, 63, 0.15)
    img = wl.make_image(64, 1, 16 + 161, 25 + 140, 3)
    monkeypatch.setenv("FRAGSCAN_POOL_FUSE", "0")
    base = _scan(fsb, layers, params, img, 3, 0, dt)
    for var, val in (("FRAGSCAN_DIRECT", "0"), ("FRAGSCAN_RUN", "0"), ("FRAGSCAN_ROWTILES", "1"),
                     ("FRAGSCAN_ROWTILES", "0")):
        monkeypatch.setenv(var, val)
        print("rect variant", dt, var, val, flush=True)
        got = _scan(fsb, layers, params, img, 3, 0, dt)
        monkeypatch.delenv(var)
        if var == "FRAGSCAN_DIRECT":
            # another first-layer kernel: another summation order
            assert np.abs(got - base).max() <= TOL[dt]
        else:
            assert np.array_equal(got, base), (var, val)
    ref = oracle.frag_cpu.frag_scan(layers, params, img, (16, 25))
    assert np.abs(base - ref).max() <= TOL[dt]


def test_rect_reassembly_bit_exact(fsb):
    """Position-encoding probe with rectangular kernels and pools: a single
    bottom-left tap per convolution and an image growing along y and x make
    every output an exact copy of one image pixel."""
    c = 2
    layers, params = [], []
    for kind, (ky, kx) in [("conv", (3, 2)), ("pool", (2, 3)), ("conv", (2, 3)), ("pool", (3, 1)),
                           ("pool", (1, 2))]:
        if kind == "pool":
            layers.append(wl.pool(ky, c, kx=kx))
            params.append(None)
        else:
            layers.append(wl.conv(ky, c, c, "none", kx=kx))
            wt = np.zeros((c, c, ky, kx), np.float32)
            for i in range(c):
                wt[i, i, ky - 1, 0] = 1.0
            params.append((wt, np.zeros(c, np.float32)))
    layers.append(wl.fc(2, c, c, "none", kx=3))
    wt = np.zeros((c, c, 2, 3), np.float32)
    for i in range(c):
        wt[i, i, 0, 2] = 1.0
    params.append((wt, np.zeros(c, np.float32)))
    h0, w0 = ix.patch_hw(layers)
    H, W = h0 + 70, w0 + 83
    yy, xx = np.meshgrid(np.arange(H), np.arange(W), indexing="ij")
    img = np.stack([yy, xx], -1)[None].astype(np.float32)
    got = _scan(fsb, layers, params, img, c)
    ref = oracle.patch_forward(layers, params, img, (h0, w0))
    assert np.array_equal(got, ref)
    ny, nx = H - h0 + 1, W - w0 + 1
    Y, X = np.meshgrid(np.arange(ny), np.arange(nx), indexing="ij")
    off_y, off_x = got[0, :, :, 0] - Y, got[0, :, :, 1] - X
    assert (off_y == off_y[0, 0]).all() and (off_x == off_x[0, 0]).all()


@pytest.mark.parametrize("mode", ["reflect", "symmetric"])
def test_rect_mirrored_borders(fsb, mode):
    """Mirrored borders with an h_0 x w_0 window: each axis extended for its
    own side; the map is H x W."""
    layers = _rect_mfma_net()
    params = wl.make_weights(layers, 65, 0.15)
    img = wl.make_image(66, 1, 41, 57, 3)
    net = fsb.Net(layers, params, 3)
    x = torch.from_numpy(img).cuda()
    got = net.scan(x, border=mode).cpu().numpy().astype(np.float64)
    net.close()
    ref = oracle.border.scan_mirrored(layers, params, img, (16, 25), mode)
    assert got.shape == ref.shape == (1, 41, 57, 2)
    assert np.abs(got - ref).max() <= TOL["f32"]


def test_rect_tiled_scan(fsb):
    """Tiled scan of the rectangular net: the untiled values bit for bit."""
    layers = _rect_mfma_net()
    params = wl.make_weights(layers, 67, 0.15)
    img = wl.make_image(68, 2, 16 + 120, 25 + 131, 3)
    net = fsb.Net(layers, params, 3)
    x = torch.from_numpy(img).cuda()
    ref = net.scan(x).cpu().numpy()
    for tile in [(37, 50), (121, 7), (1000, 1000)]:
        print("rect tiled", tile, flush=True)
        out = torch.full_like(torch.from_numpy(ref), float("nan")).cuda()
        net.scan_tiled(x, tile, out=out)
        torch.cuda.synchronize()
        assert np.array_equal(out.cpu().numpy(), ref), tile
    net.close()


@pytest.mark.parametrize("ncls", [2, 3])
def test_wide_fc_tile(fsb, monkeypatch, ncls):
    """The float32 4 x 13 register tile of a 200-output FC layer with the
    fused head (two-class and general head epilogues), forced on and off,
    against the per-patch oracle; ragged final fragments, B = 2."""
    layers = [wl.conv(3, 1, 16), wl.pool(2, 16), wl.conv(2, 16, 48), wl.pool(2, 48),
              wl.fc(3, 48, 200), wl.fc(1, 200, ncls, "softmax")]
    w0 = ix.patch_size(layers)
    params = wl.make_weights(layers, 71 + ncls, 0.1)
    img = wl.make_image(73 + ncls, 2, w0 + 95, w0 + 88, 1)
    ref = oracle.patch_forward(layers, params, img, w0)
    got = {}
    for mode in ("1", "0"):
        monkeypatch.setenv("FRAGSCAN_WIDE", mode)
        net = fsb.Net(layers, params, 1)
        names = [L["name"] for L in net.launches(2, img.shape[1], img.shape[2])]
        net.close()
        assert any(n.startswith("conv_frag_mfma<4, 13, 1, 1") for n in names) == (mode == "1"), names
        print("wide fc", ncls, mode, names[-1], flush=True)
        got[mode] = _scan(fsb, layers, params, img, 1)
        assert np.abs(got[mode] - ref).max() <= TOL["f32"]
    assert np.abs(got["1"] - got["0"]).max() <= 1e-5


def test_concurrent_streams(fsb):
    """One net, two non-default streams, distinct workspaces and outputs,
    scans enqueued on both before either is waited for: the values of
    scans run one at a time, bit for bit."""
    w = wl.WORKLOADS[2]
    params, img_a = wl.workload_inputs(2, height=230, width=210)
    img_b = wl.make_image(91, 1, 230, 210, 1)
    net = fsb.Net(w.layers, params, 1)
    xa = torch.from_numpy(img_a).cuda()
    xb = torch.from_numpy(np.ascontiguousarray(img_b)).cuda()
    ref_a = net.scan(xa).clone()
    ref_b = net.scan(xb).clone()
    torch.cuda.synchronize()
    nbytes = net.plan(1, 230, 210)["workspace_bytes"]
    ws = [torch.empty(nbytes, dtype=torch.uint8, device="cuda") for _ in range(2)]
    outs = [torch.full_like(ref_a, float("nan")) for _ in range(2)]
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    torch.cuda.synchronize()
    for _ in range(3):
        net.scan(xa, out=outs[0], workspace=ws[0], stream=s1)
        net.scan(xb, out=outs[1], workspace=ws[1], stream=s2)
    s1.synchronize()
    s2.synchronize()
    assert torch.equal(outs[0], ref_a)
    assert torch.equal(outs[1], ref_b)
    net.close()


# ---- degenerate and maximum cases of the method ----------------------------

@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_degenerate_nets(fsb, dt):
    """Stacks at the method's corners, full map against the per-patch
    oracle: a 1 x 1 pool (one child, the identity), 1 x 1 kernels only (the
    window is one pixel), a lone fully connected layer (the window is the
    whole net's input: one fragment, no pools), and an FC layer on a
    1-pixel-wide map after pools."""
    cases = [
        [wl.conv(2, 2, 3), wl.pool(1, 3), wl.conv(2, 3, 4), wl.pool(2, 4), wl.fc(2, 4, 5), wl.fc(1, 5, 2, "softmax")],
        [wl.conv(1, 3, 8), wl.conv(1, 8, 4, "none"), wl.fc(1, 4, 3, "softmax")],
        [wl.fc(7, 2, 3, "softmax")],
        [wl.conv(3, 2, 4), wl.pool(3, 4), wl.pool(2, 4), wl.fc(1, 4, 2, "softmax")],
    ]
    for n, layers in enumerate(cases):
        c0 = layers[0]["c_in"]
        w0 = ix.patch_size(layers)
        params = wl.make_weights(layers, 80 + n, 0.3)
        img = wl.make_image(90 + n, 2, w0 + 29 + n, w0 + 22, c0)
        print("degenerate", n, dt, w0, img.shape, flush=True)
        got = _scan(fsb, layers, params, img, c0, dtype=dt)
        ref = oracle.patch_forward(layers, params, img, w0)
        assert got.shape == ref.shape
        assert np.abs(got - ref).max() <= TOL[dt], n


@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_max_fragments_per_axis(fsb, dt):
    """Pools whose sizes multiply to 256 per axis, the library's limit:
    65,536 final fragments per image, most of them empty on this image,
    against the per-patch oracle on every window."""
    layers = [wl.conv(2, 1, 3), wl.pool(4, 3), wl.pool(4, 3), wl.pool(4, 3), wl.pool(4, 3),
              wl.fc(1, 3, 2, "softmax")]
    w0 = ix.patch_size(layers)
    assert w0 == 257 and ix.n_fragments(layers) == 65536
    params = wl.make_weights(layers, 95, 0.5)
    img = wl.make_image(96, 1, w0 + 43, w0 + 33, 1)
    got = _scan(fsb, layers, params, img, 1, dtype=dt)
    ref = oracle.patch_forward(layers, params, img, w0)
    assert np.abs(got - ref).max() <= TOL[dt]


# ---- pools whose stride differs from their size (overlapping, gapped) -------

@pytest.mark.parametrize("seed", [9302, 9304, 9310, 9313, 9315, 9318, 9321, 9326])
def test_stride_random_nets(fsb, seed):
    """Random stacks whose pools overlap (stride below the size) or leave
    gaps (stride above it), square and rectangular: the full map against
    the CPU fragment method and sampled windows against the per-window
    oracle; odd seeds in bf16."""
    rng = np.random.default_rng(seed)
    layers, (h0, w0), c0 = wl.random_stride_net(rng)
    dt = "bf16" if seed % 2 else "f32"
    B = 1 + seed % 2
    H, W = h0 + int(rng.integers(0, 40)), w0 + int(rng.integers(0, 40))
    params = wl.make_weights(layers, seed + 100, 0.4)
    img = wl.make_image(seed + 200, B, H, W, c0)
    print("stride net", seed, [(L["kind"], ix.kyx(L), ix.syx(L) if L["kind"] == "pool" else None)
                               for L in layers], (B, H, W), dt, flush=True)
    got = _scan(fsb, layers, params, img, c0, 0, dt)
    ref = oracle.frag_cpu.frag_scan(layers, params, img, (h0, w0))
    assert got.shape == ref.shape
    assert np.abs(got - ref).max() <= TOL[dt]
    pts = _sample_patches(layers, B, H, W, 24, seed)
    ref_p = oracle.patch_forward(layers, params, img, (h0, w0), pts)
    assert np.abs(got[pts[:, 0], pts[:, 1], pts[:, 2]] - ref_p).max() <= TOL[dt]


def _stride_mfma_net():
    """Matrix-core channel counts with an overlapping 3 x 3 pool of stride 2
    and a gapped 2 x 2 pool of stride 3; window 15 x 15, 36 final
    fragments."""
    layers = [wl.conv(3, 3, 32), wl.pool(3, 32, stride=2), wl.conv(2, 32, 48), wl.pool(2, 48, stride=3),
              wl.fc(2, 48, 24), wl.fc(1, 24, 3, "softmax")]
    assert ix.patch_hw(layers) == (15, 15) and ix.n_fragments(layers) == 36
    return layers


@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_stride_mfma_net(fsb, dt):
    """Vector-path layers around strided pools (not fused into the
    convolutions), the head fused into the last layer, two images; the full
    map against the CPU fragment method, and the tiled scan bit for bit."""
    layers = _stride_mfma_net()
    params = wl.make_weights(layers, 81, 0.15)
    img = wl.make_image(82, 2, 15 + 93, 15 + 118, 3)
    got = _scan(fsb, layers, params, img, 3, 0, dt)
    ref = oracle.frag_cpu.frag_scan(layers, params, img, 15)
    assert np.abs(got - ref).max() <= TOL[dt]
    net = fsb.Net(layers, params, 3, 0, dt)
    x = torch.from_numpy(img).cuda()
    out = torch.full((2, 94, 119, 3), float("nan"), device="cuda")
    net.scan_tiled(x, (37, 50), out=out)
    torch.cuda.synchronize()
    net.close()
    assert np.array_equal(out.cpu().numpy().astype(np.float64), got)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_stride_reassembly_bit_exact(fsb, dtype):
    """Position-encoding probe with overlapping and gapped pools: one-tap
    convolutions and an image growing along y and x make every output an
    exact copy of one image pixel (the last of each pooling window), in both
    precisions."""
    c = 3
    layers, params = [], []
    for kind, k, st in [("conv", 2, None), ("pool", 3, 2), ("conv", 2, None), ("pool", 2, 3), ("pool", 2, 1)]:
        if kind == "pool":
            layers.append(wl.pool(k, c, stride=st))
            params.append(None)
        else:
            layers.append(wl.conv(k, c, c, "none"))
            wt = np.zeros((c, c, k, k), np.float32)
            for i in range(c):
                wt[i, i, k - 1, 0] = 1.0
            params.append((wt, np.zeros(c, np.float32)))
    layers.append(wl.fc(2, c, c, "none"))
    wt = np.zeros((c, c, 2, 2), np.float32)
    for i in range(c):
        wt[i, i, 0, 1] = 1.0
    params.append((wt, np.zeros(c, np.float32)))
    h0, w0 = ix.patch_hw(layers)
    B, H, W = 2, h0 + 77, w0 + 64
    yy, xx = np.meshgrid(np.arange(H), np.arange(W), indexing="ij")
    img = np.zeros((B, H, W, c), np.float32)
    for b in range(B):
        img[b, :, :, 0] = yy % 128 + 64 * b
        img[b, :, :, 1] = xx % 128
        img[b, :, :, 2] = (yy // 128) * 16 + xx // 128 + 128 * b
    got = _scan(fsb, layers, params, img, c, dtype=dtype)
    ref = oracle.patch_forward(layers, params, img, (h0, w0))
    assert np.array_equal(got, ref)


@pytest.mark.parametrize("wid", [2, 5])
def test_pool_rows_per_thread_bit_exact(fsb, monkeypatch, wid):
    """The row-band pool kernel with 4 or 8 filter rows per thread gives the
    same values bit for bit (pools not fused, so the separate kernel runs;
    2 x 2 and 3 x 3 pools, f32 and bf16, two images)."""
    w = wl.WORKLOADS[wid]
    params, img = wl.workload_inputs(wid, batch=2, height=171, width=160)
    monkeypatch.setenv("FRAGSCAN_POOL_FUSE", "0")
    outs = {}
    for rows in ("4", "8"):
        monkeypatch.setenv("FRAGSCAN_POOL_ROWS", rows)
        net = fsb.Net(w.layers, params, w.channels, 0, w.dtype)
        names = [L["name"] for L in net.launches(2, 171, 160) if L["kind"] == 1]
        net.close()
        assert names and all(n.startswith("pool_frag_rows<") and (", %s," % rows) in n for n in names), names
        outs[rows] = _scan(fsb, w.layers, params, img, w.channels, 0, w.dtype)
    assert np.array_equal(outs["4"], outs["8"])
    ref = oracle.frag_cpu.frag_scan(w.layers, params, img, w.patch)
    assert np.abs(outs["4"] - ref).max() <= TOL[w.dtype]
