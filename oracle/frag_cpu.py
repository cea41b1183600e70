"""The fragment method on the CPU, in double precision.

TEST INFRASTRUCTURE and the CPU "image-based" baseline: see the package
docstring.  It follows Section 2.2 step by step and shares nothing with the GPU
library:

  - the image is one fragment holding the whole extended maps (Eqs. 1-2);
  - a convolutional layer keeps the fragment count and convolves every
    fragment's extended maps the way a patch is convolved, each size shrinking
    by k - 1 (Eqs. 3-4);
  - a k x k max-pooling layer turns every fragment into k^2 fragments, one per
    offset (o_x, o_y) in {0..k-1}^2; the child's pixel (xbar, ybar) is the
    maximum over o_x + k*xbar .. o_x + k*xbar + k - 1 (and the same in y) of
    the parent (Eq. 5), and its size is div(s - o, k) per axis (Eqs. 6-7);
    children of fragment f are numbered f*k^2 + o_y*k + o_x;
  - fully connected layers act on every fragment as convolutions whose kernel
    covers the whole patch-level map (Section 3: a fragment depends on one
    fragment of the layer below, for fully connected layers too);
  - the last layer's softmax is taken per pixel over the classes.

Every fragment carries where its pixel (0, 0) lands in the output and the step
between its neighbouring pixels: the input fragment starts at (0, 0) with step
1; the child at offset o of a fragment with base b and step t gets base
b + o*t and step t*k, since its window xbar starts at parent pixel o + k*xbar
(per axis: with a k_y x k_x pool, Section 2's rectangular case, the steps of
the two axes differ).  A pool whose stride s differs from its size k (not in
the paper, whose pools do not overlap) has s^2 children per fragment, one per
offset o in {0..s-1}^2, child pixel xbar covering parent pixels
o + s*xbar .. o + s*xbar + k - 1: base b + o*t and step t*s.
A fragment pixel (y, x) at the end is the patch whose top-left corner is
(base_y + step*y, base_x + step*x): a crop of a fragment's maps is one patch's
maps (Section 3).
"""
import numpy as np


def _conv(a, w, b, act):
    """Valid cross-correlation of one fragment a [h, w, ci] with OIHW weights."""
    co, ci, ky, kx = w.shape
    h, wd, _ = a.shape
    ho, wo = max(h - ky + 1, 0), max(wd - kx + 1, 0)
    out = np.empty((ho, wo, co), np.float64)
    out[...] = b
    if ho and wo:
        for dy in range(ky):
            for dx in range(kx):
                out += a[dy:dy + ho, dx:dx + wo, :] @ w[:, :, dy, dx].T
    if act == "tanh":
        np.tanh(out, out=out)
    return out


def _pool_children(a, ky, kx, sy, sx):
    """The sy*sx children of fragment a [h, w, c] under a ky x kx pool with
    stride (sy, sx), in offset order (o_y, o_x): child pixel (ybar, xbar) is
    the maximum over rows o_y + sy*ybar .. + ky - 1 and columns
    o_x + sx*xbar .. + kx - 1, for every window that ends inside a."""
    h, wd, c = a.shape
    kids = []
    for oy in range(sy):
        for ox in range(sx):
            hc, wc = max(h - oy - ky + sy, 0) // sy, max(wd - ox - kx + sx, 0) // sx
            m = np.full((hc, wc, c), -np.inf)
            for i in range(ky):
                for j in range(kx):
                    y0, x0 = oy + i, ox + j
                    m = np.maximum(m, a[y0:y0 + sy * hc:sy, x0:x0 + sx * wc:sx, :][:hc, :wc])
            kids.append(((oy, ox), m))
    return kids


def frag_scan(layers, params, image, patch):
    """Outputs of the net for every patch of every image, [B, H-h0+1, W-w0+1, n]
    (patch: w_0, or (h_0, w_0))."""
    img = np.asarray(image, dtype=np.float64)
    B, H, W, C = img.shape
    h0, w0 = (patch, patch) if np.isscalar(patch) else patch
    ny, nx = H - h0 + 1, W - w0 + 1
    n_out = layers[-1]["c_out"]
    res = np.full((B, ny, nx, n_out), np.nan)
    for b in range(B):
        # (base_y, base_x, step_y, step_x, maps)
        frags = [(0, 0, 1, 1, img[b])]
        for L, p in zip(layers, params):
            if L["kind"] == "pool":
                ky, kx = L["k"], L.get("kx", L["k"])
                sy = L.get("stride", ky)
                sx = L.get("stride_x", sy if "stride" in L else kx)
                nxt = []
                for (by, bx, ty, tx, a) in frags:
                    for (oy, ox), m in _pool_children(a, ky, kx, sy, sx):
                        nxt.append((by + oy * ty, bx + ox * tx, ty * sy, tx * sx, m))
                frags = nxt
            else:
                w = np.asarray(p[0], np.float64)
                bias = np.asarray(p[1], np.float64)
                frags = [(by, bx, ty, tx, _conv(a, w, bias, L["act"])) for (by, bx, ty, tx, a) in frags]
        for (by, bx, ty, tx, a) in frags:
            z = a
            if layers[-1]["act"] == "softmax" and z.size:
                z = z - z.max(axis=-1, keepdims=True)
                z = np.exp(z)
                z = z / z.sum(axis=-1, keepdims=True)
            hf, wf = z.shape[:2]
            res[b, by:by + ty * hf:ty, bx:bx + tx * wf:tx, :] = z
    return res
