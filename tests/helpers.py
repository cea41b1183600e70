"""Test-side helpers: an independent whole-map formulation and random nets."""
import numpy as np
import torch
import torch.nn.functional as F


def _k(L):
    """(rows, columns) of a layer's kernel or pool."""
    return L["k"], L.get("kx", L["k"])


def _s(L):
    """(rows, columns) stride of a pool (its size unless given)."""
    ky, kx = _k(L)
    sy = L.get("stride", ky)
    return sy, L.get("stride_x", sy if "stride" in L else kx)


def torch_patch_net(layers, params, crop):
    """The net on one patch with torch CPU library routines, float64.
    crop: [h0, w0, C] -> returns [n_out]."""
    x = torch.from_numpy(np.asarray(crop, np.float64)).permute(2, 0, 1)[None]
    for L, p in zip(layers, params):
        if L["kind"] == "pool":
            x = F.max_pool2d(x, _k(L), stride=_s(L))
        else:
            w = torch.from_numpy(np.asarray(p[0], np.float64))
            b = torch.from_numpy(np.asarray(p[1], np.float64))
            if L["kind"] == "fc":
                assert (x.shape[-2], x.shape[-1]) == _k(L)
                x = F.linear(x.reshape(1, -1), w.reshape(w.shape[0], -1), b)[:, :, None, None]
            else:
                x = F.conv2d(x, w, b)
            if L["act"] == "tanh":
                x = torch.tanh(x)
    z = x.reshape(-1)
    if layers[-1]["act"] == "softmax":
        z = torch.softmax(z, 0)
    return z.numpy()


def dilated_scan(layers, params, image):
    """Whole-map formulation with dilated library convolutions: a conv after
    pools of cumulative stride S is a convolution with dilation S, a k-pool is
    a stride-1 max-pool with dilation S, and then S grows by the pool's stride
    (its size k unless it has another; per axis).
    Output index = patch top-left corner.  [B,H,W,C] -> [B, H-h0+1, W-w0+1, n]."""
    x = torch.from_numpy(np.asarray(image, np.float64)).permute(0, 3, 1, 2)
    Sy = Sx = 1
    for L, p in zip(layers, params):
        ky, kx = _k(L)
        if L["kind"] == "pool":
            x = F.max_pool2d(x, (ky, kx), stride=1, dilation=(Sy, Sx))
            Sy *= _s(L)[0]
            Sx *= _s(L)[1]
        else:
            w = torch.from_numpy(np.asarray(p[0], np.float64))
            b = torch.from_numpy(np.asarray(p[1], np.float64))
            x = F.conv2d(x, w, b, dilation=(Sy, Sx))
            if L["act"] == "tanh":
                x = torch.tanh(x)
    if layers[-1]["act"] == "softmax":
        x = torch.softmax(x, 1)
    return x.permute(0, 2, 3, 1).numpy()
