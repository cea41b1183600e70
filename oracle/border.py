"""Mirrored image borders (Section 3.2: the edges of the 512 x 512 slice are
mirrored so that the net can be applied at every position).  TEST
INFRASTRUCTURE, like the rest of this package.

The paper does not say how the edges are mirrored or how an even patch is
centred.  Readings:
  - the image is extended by p0 = floor((w_0 - 1) / 2) pixels before the first
    row / column and w_0 - 1 - p0 after the last, so that the window with
    top-left (y, x) of the extended image is centred on image pixel (y, x)
    (for even w_0: the pixel p0 below and right of its top-left) and the
    output map is H x W;
  - "reflect" mirrors about the edge pixels (..., 2, 1, | 0, 1, 2, ...),
    "symmetric" repeats them (..., 1, 0, | 0, 1, ...), both repeatedly for
    borders wider than the image: numpy's pad modes of the same names.
"""
import numpy as np

from .patch import patch_forward

MODES = ("reflect", "symmetric")


def border_widths(patch):
    """(before, after) extension of each axis for a w_0 x w_0 window."""
    p0 = (patch - 1) // 2
    return p0, patch - 1 - p0


def mirror_pad(image, patch, mode):
    """[B, H, W, C] image -> [B, H + h_0 - 1, W + w_0 - 1, C] extended image
    (patch: w_0, or (h_0, w_0); each axis is extended for its own side)."""
    if mode not in MODES:
        raise ValueError("mode must be one of %s" % (MODES,))
    h0, w0 = (patch, patch) if np.isscalar(patch) else patch
    (ly, hy), (lx, hx) = border_widths(h0), border_widths(w0)
    return np.pad(np.asarray(image, np.float64), ((0, 0), (ly, hy), (lx, hx), (0, 0)), mode=mode)


def scan_mirrored(layers, params, image, patch, mode, patches=None):
    """The net on every window of the extended image (all H x W outputs, or
    the requested (b, y, x) ones), in float64: output (b, y, x) is the window
    centred on image pixel (y, x)."""
    return patch_forward(layers, params, mirror_pad(image, patch, mode), patch, patches)
