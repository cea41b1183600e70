"""ctypes wrapper of the per-patch oracle (patch_oracle.c).

TEST INFRASTRUCTURE: see the package docstring.  Follows Section 2.1 of the
paper (patch-level testing) and the output set of Section 2.2 (every window of
size w_0 inside the image).
"""
import ctypes
import os

import numpy as np

from . import build as _build

ORACLE_LIB = _build.LIB
_lib = None

KIND = {"conv": 0, "pool": 1, "fc": 2}
ACT = {"none": 0, "tanh": 1, "softmax": 2}


class _OLayer(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int), ("k", ctypes.c_int), ("kx", ctypes.c_int), ("c_in", ctypes.c_int),
                ("c_out", ctypes.c_int), ("act", ctypes.c_int),
                ("w", ctypes.POINTER(ctypes.c_double)),
                ("b", ctypes.POINTER(ctypes.c_double)),
                ("s", ctypes.c_int), ("sx", ctypes.c_int)]


def _open(path):
    lib = ctypes.CDLL(path)
    lib.oracle_patch_forward.restype = ctypes.c_int
    lib.oracle_patch_forward.argtypes = [
        ctypes.POINTER(_OLayer), ctypes.c_int, ctypes.POINTER(ctypes.c_double),
        ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int,
        ctypes.POINTER(ctypes.c_int), ctypes.c_long, ctypes.POINTER(ctypes.c_double)]
    return lib


def _load(path=None):
    """The compiled oracle (built on first use); `path` loads another build of
    the same source, which the planted-mistake tests use."""
    global _lib
    if path is not None:
        return _open(path)
    if _lib is None:
        if not os.path.exists(ORACLE_LIB):
            _build.build(force=True, quiet=True)
        _lib = _open(ORACLE_LIB)
    return _lib


def _dptr(a):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_double))


def patch_forward(layers, params, image, patch, patches=None, lib_path=None):
    """Outputs of the net on the requested patches, in float64.

    layers  : layer dicts (kind, k, c_in, c_out, act; optional kx, the
              kernel's / pool's columns when they differ from its rows k;
              pools: optional stride, stride_x when they differ from k, kx)
    params  : per layer (weight OIHW, bias) or None for pools
    image   : [B][H][W][C] array (any float type; promoted to float64)
    patch   : w_0, or (h_0, w_0) for a rectangular window
    patches : int array [n, 3] of (b, Y, X) top-left corners; None = all of them
    Returns [n, n_out] float64, or, when patches is None, [B, H-h0+1, W-w0+1, n_out].
    """
    lib = _load(lib_path)
    h0, w0 = (patch, patch) if np.isscalar(patch) else (int(patch[0]), int(patch[1]))
    img = np.ascontiguousarray(image, dtype=np.float64)
    B, H, W, C = img.shape
    keep = []
    arr = (_OLayer * len(layers))()
    for i, (L, p) in enumerate(zip(layers, params)):
        arr[i].kind, arr[i].k, arr[i].kx = KIND[L["kind"]], L["k"], L.get("kx", 0)
        arr[i].c_in, arr[i].c_out, arr[i].act = L["c_in"], L["c_out"], ACT[L["act"]]
        arr[i].s, arr[i].sx = L.get("stride", 0), L.get("stride_x", 0)
        if p is not None:
            w = np.ascontiguousarray(p[0], dtype=np.float64)
            b = np.ascontiguousarray(p[1], dtype=np.float64)
            keep += [w, b]
            arr[i].w, arr[i].b = _dptr(w), _dptr(b)
    full = patches is None
    if full:
        ny, nx = H - h0 + 1, W - w0 + 1
        bb, yy, xx = np.meshgrid(np.arange(B), np.arange(ny), np.arange(nx), indexing="ij")
        patches = np.stack([bb.ravel(), yy.ravel(), xx.ravel()], axis=1)
    patches = np.ascontiguousarray(patches, dtype=np.int32)
    n = patches.shape[0]
    n_out = layers[-1]["c_out"]
    out = np.zeros((n, n_out), np.float64)
    rc = lib.oracle_patch_forward(arr, len(layers), _dptr(img), B, H, W, C, h0, w0,
                                  patches.ctypes.data_as(ctypes.POINTER(ctypes.c_int)),
                                  n, _dptr(out))
    if rc != 0:
        raise ValueError("oracle: invalid net, patch size or patch list")
    if full:
        return out.reshape(B, H - h0 + 1, W - w0 + 1, n_out)
    return out
