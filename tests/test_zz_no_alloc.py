"""fs_scan_noalloc (no workspace argument, no device allocation) through the
C-ABI against fs_scan: the same kernels and plan on the library's per-GPU
scratch array, so the same outputs bit for bit, on two calls in a row, the
second with a smaller image (the array keeps the first call's contents)."""
import ctypes

import numpy as np
import pytest

import oracle
from paper_1302_1700_amd import workloads as wl

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def fsb():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_1302_1700_amd import fragscan
    fragscan.load()
    return fragscan


def _noalloc(fsb, net, x):
    B, H, W, _ = x.shape
    out = torch.full((B, H - net.patch + 1, W - net.patch_x + 1, net.n_classes), float("nan"), device=x.device)
    lib = fsb.load()
    st = lib.fs_scan_noalloc(net._h, ctypes.c_void_p(x.data_ptr()), B, H, W, ctypes.c_void_p(out.data_ptr()),
                             ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
    assert st == fsb.FS_OK, lib.fs_last_error()
    torch.cuda.synchronize()
    return out


@pytest.mark.parametrize("wid,sizes", [(2, [(1, 512, 512), (1, 200, 171)]),
                                       (5, [(1, 300, 280), (1, 97, 120)]),
                                       (1, [(2, 64, 64), (1, 20, 33)])])
def test_noalloc_matches_scan(fsb, wid, sizes):
    w = wl.WORKLOADS[wid]
    params, _ = wl.workload_inputs(wid, height=w.patch, width=w.patch)
    net = fsb.Net(w.layers, params, w.channels, 0, w.dtype)
    for n, (B, H, W) in enumerate(sizes):
        print("noalloc", wid, (B, H, W), flush=True)
        img = wl.make_image(300 + 10 * wid + n, B, H, W, w.channels)
        x = torch.from_numpy(img).cuda()
        ref = net.scan(x).clone()
        torch.cuda.synchronize()
        got = _noalloc(fsb, net, x)
        assert torch.equal(got, ref), (wid, B, H, W)
        if n == len(sizes) - 1:
            pts = np.array([(b, y, x_) for b in range(B) for y in (0, H - w.patch) for x_ in (0, W - w.patch)],
                           np.int32)
            want = oracle.patch_forward(w.layers, params, img, w.patch, pts)
            g = got.cpu().numpy().astype(np.float64)[pts[:, 0], pts[:, 1], pts[:, 2]]
            assert np.abs(g - want).max() <= (2e-2 if w.dtype == "bf16" else 1e-4)
    net.close()


def test_noalloc_refuses_large_scan(fsb):
    w = wl.WORKLOADS[2]
    params, _ = wl.workload_inputs(2, height=95, width=95)
    net = fsb.Net(w.layers, params, 1)
    x = torch.zeros((1, 1024, 1024, 1), device="cuda")
    out = torch.empty((1, 930, 930, 2), device="cuda")
    with pytest.raises(fsb.FsError) as e:
        net.scan_noalloc(x, out)
    assert e.value.status == fsb.FS_ERR_WORKSPACE
    net.close()
