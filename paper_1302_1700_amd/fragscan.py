"""Python binding of libfragscan.so (include/fragscan.h).

Argument marshalling only: PyTorch supplies device memory and the current
stream; every step of the scan runs in the library's HIP kernels.  Names mirror
the C entry points (fs_net_create -> Net, fs_scan -> Net.scan, ...).
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libfragscan.so")
# the same library with the kernels' bounds checks compiled in (FS_ERR_BOUNDS)
LIB_DEBUG_PATH = os.path.join(_HERE, "libfragscan_debug.so")

(FS_OK, FS_ERR_INVALID_ARG, FS_ERR_SHAPE, FS_ERR_UNSUPPORTED, FS_ERR_WORKSPACE, FS_ERR_OOM, FS_ERR_HIP,
 FS_ERR_BOUNDS) = range(8)
KIND = {"conv": 0, "pool": 1, "fc": 2}
ACT = {"none": 0, "tanh": 1, "softmax": 2}
DTYPE = {"f32": 0, "bf16": 1}
BORDER = {"valid": 0, "reflect": 1, "symmetric": 2}


class FsError(RuntimeError):
    def __init__(self, status, msg):
        super().__init__("fragscan status %d: %s" % (status, msg))
        self.status = status


class fs_layer(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int32), ("k", ctypes.c_int32), ("c_in", ctypes.c_int32),
                ("c_out", ctypes.c_int32), ("act", ctypes.c_int32),
                ("weight", ctypes.c_void_p), ("bias", ctypes.c_void_p), ("k_x", ctypes.c_int32),
                ("stride", ctypes.c_int32), ("stride_x", ctypes.c_int32)]


class fs_net_info(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in ("patch", "in_channels", "n_classes", "n_layers",
                                              "n_pools", "stride", "n_fragments", "dtype",
                                              "patch_x", "stride_x")]


class fs_plan_info(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("out_h", ctypes.c_int32), ("out_w", ctypes.c_int32),
                ("n_launches", ctypes.c_int32), ("workspace_bytes", ctypes.c_size_t),
                ("flops", ctypes.c_double), ("min_bytes", ctypes.c_double)]


class fs_launch_info(ctypes.Structure):
    _fields_ = [("layer", ctypes.c_int32), ("n_layers", ctypes.c_int32), ("kind", ctypes.c_int32),
                ("fragments", ctypes.c_int32), ("out_pixels", ctypes.c_int64),
                ("flops", ctypes.c_double), ("bytes", ctypes.c_double),
                ("grid", ctypes.c_int32), ("block", ctypes.c_int32), ("name", ctypes.c_char * 96),
                ("lds_bytes", ctypes.c_int32), ("per_cu", ctypes.c_int32)]


EXPORTS = ["fs_net_create", "fs_net_create_plan_only", "fs_net_destroy", "fs_net_query", "fs_scan_plan", "fs_scan_launches",
           "fs_scan", "fs_scan_profile", "fs_fragment_table", "fs_reassembly_index",
           "fs_status_str", "fs_last_error", "fs_scan_plan_border", "fs_scan_border",
           "fs_scan_plan_tiled", "fs_scan_tiled", "fs_scan_noalloc"]

_libs = {}


def load(debug=False):
    """Load libfragscan.so (debug=True: libfragscan_debug.so); raises if it
    has not been built (no fallback)."""
    if debug in _libs:
        return _libs[debug]
    path = LIB_DEBUG_PATH if debug else LIB_PATH
    if not os.path.exists(path):
        raise RuntimeError("%s is not built; run __graft_entry__.build() or "
                           "python paper_1302_1700_amd/build.py" % path)
    lib = ctypes.CDLL(path)
    P, I32, SZ, VP = ctypes.POINTER, ctypes.c_int32, ctypes.c_size_t, ctypes.c_void_p
    sig = {
        "fs_net_create": [P(fs_layer), I32, I32, I32, I32, P(VP)],
        "fs_net_create_plan_only": [P(fs_layer), I32, I32, I32, I32, P(VP)],
        "fs_net_destroy": [VP],
        "fs_net_query": [VP, P(fs_net_info)],
        "fs_scan_plan": [VP, I32, I32, I32, P(fs_plan_info)],
        "fs_scan_plan_border": [VP, I32, I32, I32, I32, P(fs_plan_info)],
        "fs_scan_border": [VP, VP, I32, I32, I32, I32, VP, VP, SZ, VP],
        "fs_scan_plan_tiled": [VP, I32, I32, I32, I32, I32, P(fs_plan_info)],
        "fs_scan_tiled": [VP, VP, I32, I32, I32, I32, I32, VP, VP, SZ, VP],
        "fs_scan_launches": [VP, I32, I32, I32, P(fs_launch_info), I32],
        "fs_scan": [VP, VP, I32, I32, I32, VP, VP, SZ, VP],
        "fs_scan_noalloc": [VP, VP, I32, I32, I32, VP, VP],
        "fs_scan_profile": [VP, VP, I32, I32, I32, VP, VP, SZ, VP, I32, P(ctypes.c_float), I32],
        "fs_fragment_table": [VP, I32, I32, P(I32), SZ, P(SZ)],
        "fs_reassembly_index": [VP, I32, I32, P(I32), SZ, P(SZ)],
        "fs_status_str": [ctypes.c_int],
        "fs_last_error": [],
    }
    for name, args in sig.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = ctypes.c_int
    lib.fs_net_destroy.restype = None
    lib.fs_status_str.restype = ctypes.c_char_p
    lib.fs_last_error.restype = ctypes.c_char_p
    _libs[debug] = lib
    return lib


def _check(st, lib=None):
    if st != FS_OK:
        lib = lib or load()
        raise FsError(st, lib.fs_last_error().decode())


def check_tensors(image, out, workspace, in_channels, out_shape, require_cuda=True):
    """Argument checks done before any pointer reaches the library, which
    only sees addresses and sizes: the image must be a contiguous float32
    [B, H, W, in_channels] tensor (on a GPU unless require_cuda is False);
    `out`, when given, a contiguous float32 tensor of exactly out_shape on
    the image's device; `workspace`, when given, a contiguous tensor on the
    image's device.  Raises ValueError."""
    import torch
    if image.dim() != 4 or image.dtype != torch.float32 or not image.is_contiguous():
        raise ValueError("image must be a contiguous float32 tensor [B, H, W, C]")
    if require_cuda and not image.is_cuda:
        raise ValueError("image must be on a GPU")
    if image.shape[3] != in_channels:
        raise ValueError("image has %d channels, the net takes %d" % (image.shape[3], in_channels))
    if out is not None:
        if out.dtype != torch.float32 or not out.is_contiguous():
            raise ValueError("out must be a contiguous float32 tensor")
        if tuple(out.shape) != tuple(out_shape):
            raise ValueError("out has shape %s, the scan writes %s" % (tuple(out.shape), tuple(out_shape)))
        if out.device != image.device:
            raise ValueError("out is on %s, the image on %s" % (out.device, image.device))
    if workspace is not None:
        if not workspace.is_contiguous():
            raise ValueError("workspace must be contiguous")
        if workspace.device != image.device:
            raise ValueError("workspace is on %s, the image on %s" % (workspace.device, image.device))


def _nbytes(t):
    return t.numel() * t.element_size()


def _stream_handle(stream=None):
    import torch
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


class Net:
    """A net loaded into the library.

    layers : list of layer dicts (kind, k, c_in, c_out, act; optional kx, the
             kernel's / pool's columns when they differ from its rows k;
             pools: optional stride, stride_x), see workloads.py
    params : per layer (weight OIHW float32, bias float32) or None for pools
    in_channels, patch (0 = derive), dtype "f32" | "bf16".
    Created on the current HIP device; plan_only=True makes a host-only handle
    for planning and index queries (no device needed, cannot scan); debug=True
    loads the net into libfragscan_debug.so, whose kernels check every fragment
    access (a failed check raises FsError with status FS_ERR_BOUNDS).
    """

    def __init__(self, layers, params, in_channels, patch=0, dtype="f32", plan_only=False, debug=False):
        lib = self._lib = load(debug)
        self._keep = []
        arr = (fs_layer * len(layers))()
        for i, (L, p) in enumerate(zip(layers, params)):
            arr[i].kind = KIND[L["kind"]]
            arr[i].k = int(L["k"])
            arr[i].k_x = int(L.get("kx") or 0)
            arr[i].stride = int(L.get("stride") or 0)
            arr[i].stride_x = int(L.get("stride_x") or 0)
            arr[i].c_in = int(L["c_in"])
            arr[i].c_out = int(L["c_out"])
            arr[i].act = ACT[L["act"]]
            if p is not None:
                w = np.ascontiguousarray(p[0], dtype=np.float32)
                b = np.ascontiguousarray(p[1], dtype=np.float32) if p[1] is not None else None
                self._keep += [w, b]
                arr[i].weight = w.ctypes.data
                arr[i].bias = b.ctypes.data if b is not None else None
        h = ctypes.c_void_p()
        create = lib.fs_net_create_plan_only if plan_only else lib.fs_net_create
        _check(create(arr, len(layers), int(in_channels), int(patch), DTYPE[dtype], ctypes.byref(h)), self._lib)
        self._h = h
        self._keep = None
        self._ws = {}
        info = fs_net_info()
        _check(lib.fs_net_query(self._h, ctypes.byref(info)), self._lib)
        self.info = {n: getattr(info, n) for n, _ in fs_net_info._fields_}
        self.patch = self.info["patch"]      # window rows h_0
        self.patch_x = self.info["patch_x"]  # window columns w_0
        self.n_classes = self.info["n_classes"]

    def close(self):
        if getattr(self, "_h", None):
            self._lib.fs_net_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    # -- planning --------------------------------------------------------------
    def plan(self, B, H, W, border="valid"):
        p = fs_plan_info()
        if border == "valid":
            _check(self._lib.fs_scan_plan(self._h, B, H, W, ctypes.byref(p)), self._lib)
        else:
            _check(self._lib.fs_scan_plan_border(self._h, B, H, W, BORDER[border], ctypes.byref(p)), self._lib)
        return {n: getattr(p, n) for n, _ in fs_plan_info._fields_}

    def launches(self, B, H, W):
        n = self.plan(B, H, W)["n_launches"]
        arr = (fs_launch_info * n)()
        _check(self._lib.fs_scan_launches(self._h, B, H, W, arr, n), self._lib)
        out = []
        for a in arr:
            d = {n_: getattr(a, n_) for n_, _ in fs_launch_info._fields_}
            d["name"] = a.name.decode()
            out.append(d)
        return out

    def fragment_table(self, H, W):
        lib = self._lib
        need = ctypes.c_size_t()
        _check(lib.fs_fragment_table(self._h, H, W, None, 0, ctypes.byref(need)), self._lib)
        buf = np.zeros(need.value, np.int32)
        _check(lib.fs_fragment_table(self._h, H, W, buf.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)),
                                     need.value, None), self._lib)
        rec = 5 + 2 * self.info["n_pools"]
        return buf.reshape(-1, rec)

    def reassembly_index(self, H, W):
        lib = self._lib
        need = ctypes.c_size_t()
        _check(lib.fs_reassembly_index(self._h, H, W, None, 0, ctypes.byref(need)), self._lib)
        buf = np.zeros(need.value, np.int32)
        _check(lib.fs_reassembly_index(self._h, H, W, buf.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)),
                                       need.value, None), self._lib)
        return buf.reshape(H - self.patch + 1, W - self.patch_x + 1, 3)

    # -- scanning --------------------------------------------------------------
    def plan_tiled(self, B, H, W, tile):
        """Plan of scan_tiled with output tiles of tile = (rows, cols) windows."""
        p = fs_plan_info()
        _check(self._lib.fs_scan_plan_tiled(self._h, B, H, W, int(tile[0]), int(tile[1]), ctypes.byref(p)),
                                            self._lib)
        return {n: getattr(p, n) for n, _ in fs_plan_info._fields_}

    def workspace(self, B, H, W, device=None, border="valid", tile=None):
        import torch
        nbytes = (self.plan_tiled(B, H, W, tile) if tile else self.plan(B, H, W, border))["workspace_bytes"]
        key = (nbytes, str(device))
        ws = self._ws.get(key)
        if ws is None:
            self._ws.clear()
            ws = torch.empty(max(nbytes, 256), dtype=torch.uint8, device=device or "cuda")
            self._ws[key] = ws
        return ws

    def scan(self, image, out=None, workspace=None, stream=None, border="valid"):
        """image: CUDA float32 tensor [B, H, W, C] (contiguous) -> [B, H-h0+1, W-w0+1, n]
        (border "valid"), or [B, H, W, n] with the image's edges mirrored
        ("reflect": about the edge pixels, "symmetric": edge pixels repeated)."""
        import torch
        if border not in BORDER:
            raise ValueError("border must be one of %s" % sorted(BORDER))
        if image.dim() != 4:
            raise ValueError("image must be [B, H, W, C]")
        B, H, W, C = image.shape
        oh, ow = (H - self.patch + 1, W - self.patch_x + 1) if border == "valid" else (H, W)
        check_tensors(image, out, workspace, self.info["in_channels"], (B, oh, ow, self.n_classes))
        if out is None:
            out = torch.empty((B, oh, ow, self.n_classes), dtype=torch.float32, device=image.device)
        ws = workspace if workspace is not None else self.workspace(B, H, W, image.device, border)
        if border == "valid":
            _check(self._lib.fs_scan(self._h, ctypes.c_void_p(image.data_ptr()), B, H, W,
                                     ctypes.c_void_p(out.data_ptr()), ctypes.c_void_p(ws.data_ptr()),
                                     _nbytes(ws), _stream_handle(stream)), self._lib)
        else:
            _check(self._lib.fs_scan_border(self._h, ctypes.c_void_p(image.data_ptr()), B, H, W, BORDER[border],
                                            ctypes.c_void_p(out.data_ptr()), ctypes.c_void_p(ws.data_ptr()),
                                            _nbytes(ws), _stream_handle(stream)), self._lib)
        return out

    def scan_noalloc(self, image, out, stream=None):
        """As scan (valid windows) through fs_scan_noalloc: no workspace, no
        device allocation in the call (the library's per-GPU scratch array;
        calls overlapping on one GPU race).  `out` is required."""
        if image.dim() != 4:
            raise ValueError("image must be [B, H, W, C]")
        B, H, W, C = image.shape
        shape = (B, H - self.patch + 1, W - self.patch_x + 1, self.n_classes)
        if out is None:
            raise ValueError("scan_noalloc writes into a given output tensor")
        check_tensors(image, out, None, self.info["in_channels"], shape)
        _check(self._lib.fs_scan_noalloc(self._h, ctypes.c_void_p(image.data_ptr()), B, H, W,
                                         ctypes.c_void_p(out.data_ptr()), _stream_handle(stream)), self._lib)
        return out

    def scan_tiled(self, image, tile, out=None, workspace=None, stream=None):
        """As scan (valid windows), computed tile by tile: output tiles of at
        most tile = (rows, cols) windows, each a fragment scan of the image
        region it covers, sharing one workspace sized for a tile."""
        import torch
        if image.dim() != 4:
            raise ValueError("image must be [B, H, W, C]")
        B, H, W, C = image.shape
        shape = (B, H - self.patch + 1, W - self.patch_x + 1, self.n_classes)
        check_tensors(image, out, workspace, self.info["in_channels"], shape)
        if out is None:
            out = torch.empty(shape, dtype=torch.float32, device=image.device)
        ws = workspace if workspace is not None else self.workspace(B, H, W, image.device, tile=tile)
        _check(self._lib.fs_scan_tiled(self._h, ctypes.c_void_p(image.data_ptr()), B, H, W, int(tile[0]), int(tile[1]),
                                       ctypes.c_void_p(out.data_ptr()), ctypes.c_void_p(ws.data_ptr()), _nbytes(ws),
                                       _stream_handle(stream)), self._lib)
        return out

    def profile(self, image, reps=10, out=None, stream=None):
        """Per-launch mean duration in milliseconds: each launch runs `reps`
        times back to back between two HIP events on the stream
        (synchronises; `out` ends as after one scan)."""
        import torch
        if image.dim() != 4:
            raise ValueError("image must be [B, H, W, C]")
        B, H, W, C = image.shape
        shape = (B, H - self.patch + 1, W - self.patch_x + 1, self.n_classes)
        check_tensors(image, out, None, self.info["in_channels"], shape)
        if out is None:
            out = torch.empty(shape, dtype=torch.float32, device=image.device)
        ws = self.workspace(B, H, W, image.device)
        n = self.plan(B, H, W)["n_launches"]
        ms = (ctypes.c_float * n)()
        _check(self._lib.fs_scan_profile(self._h, ctypes.c_void_p(image.data_ptr()), B, H, W,
                                         ctypes.c_void_p(out.data_ptr()), ctypes.c_void_p(ws.data_ptr()),
                                         _nbytes(ws), _stream_handle(stream), reps, ms, n), self._lib)
        return list(ms)
