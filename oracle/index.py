"""Index side of the oracle: sizes, fragment bookkeeping and FLOP counts.

TEST INFRASTRUCTURE: see the package docstring.  Everything here is plain
integer arithmetic written from the paper:

  patch_sizes       patch-level map sizes w_l (Section 2.1.1: conv gives
                    w - (k - 1); Section 2.1.2: pool gives w / k and needs
                    mod(w, k) = 0)
  patch_size        the w_0 a stack implies (last map 1 x 1)
  track             brute-force tracking of a patch's top-left corner through
                    the layers (convs keep it, a k-pool at corner x selects the
                    child with offset x mod k at position x div k, because that
                    child's windows start at o + k*xbar, Eq. 5); gives the
                    final fragment id and the position inside it
  fragment_extents  the fragments of every layer with their sizes from
                    Eqs. 1-4 and 6-7; children of a fragment are numbered
                    parent*k^2 + o_y*k + o_x, the order of the offset list in
                    Section 2.2.2 (o_x varies fastest); div is floor division
                    and a size never goes below 0

Section 2 writes all of it for square maps and kernels and notes that
rectangular ones follow directly: a layer's "k" is its rows (the y axis) and
its optional "kx" its columns; every rule above then holds per axis (a
k_y x k_x pool has k_y * k_x children, numbered parent*k_y*k_x + o_y*k_x +
o_x).

Pools whose stride s differs from their size k (optional "stride",
"stride_x"; the paper's pools are non-overlapping, s = k) generalise the same
way: at patch level a side w gives (w - k) / s + 1 (requiring (w - k) mod s
= 0); in the fragment method a fragment has s^2 children, one per offset o in
{0..s-1}^2, child pixel xbar taking the maximum over o + s*xbar ..
o + s*xbar + k - 1 (Eq. 5 with the window start stepping by s), so the child
holds div(s_f - o - k + s, s) pixels per axis (Eqs. 6-7: the windows starting
at o, o + s, ... that end inside the fragment), and tracking a corner x
through the pool selects offset x mod s at position x div s.
  fragment_table    per final fragment: offsets, base output pixel, size,
                    all found by tracking every output pixel
  reassembly_index  per output pixel: (f, y_f, x_f), by tracking
  flops_patch / flops_image   the two formulas of Section 3.1 (Table 2)
  algorithmic_flops exact multiply-add count of the scan: 2 * c_in * k^2 *
                    c_out (k_y * k_x for a rectangular kernel) per output
                    pixel of every fragment, summed
"""
import numpy as np


def kyx(L):
    """(rows, columns) of a layer's kernel or pool."""
    return L["k"], L.get("kx", L["k"])


def syx(L):
    """(rows, columns) stride of a pool: its size unless given; a column
    stride that is not given follows the row stride when that one is."""
    ky, kx = kyx(L)
    sy = L.get("stride", ky)
    return sy, L.get("stride_x", sy if "stride" in L else kx)


def patch_sizes(layers, w0, axis=0):
    """[w_0, w_1, ..., w_n] along one axis (0: rows, 1: columns) for a patch
    of that size; raises on a pool that does not divide its map or a kernel
    larger than its map."""
    sizes = [w0]
    w = w0
    for L in layers:
        k = kyx(L)[axis]
        if L["kind"] == "pool":
            st = syx(L)[axis]
            if w < k or (w - k) % st:
                raise ValueError("pool %d (stride %d) does not tile map %d" % (k, st, w))
            w = (w - k) // st + 1
        else:
            if k > w:
                raise ValueError("kernel %d larger than map %d" % (k, w))
            w -= k - 1
        sizes.append(w)
    return sizes


def patch_size(layers, axis=0):
    """w_0 implied by the stack along one axis: walk down from a 1 x 1 final
    map."""
    w = 1
    for L in reversed(layers):
        k = kyx(L)[axis]
        w = (w - 1) * syx(L)[axis] + k if L["kind"] == "pool" else w + k - 1
    return w


def patch_hw(layers):
    """(h_0, w_0): the window of a stack with rectangular kernels or pools."""
    return patch_size(layers, 0), patch_size(layers, 1)


def track(layers, Y, X):
    """Vectorised over numpy arrays Y, X of patch corners.
    Returns (f, y, x, offsets) with offsets a list, per pool, of (o_x, o_y)."""
    f = np.zeros_like(Y)
    y = np.array(Y, copy=True)
    x = np.array(X, copy=True)
    offs = []
    for L in layers:
        if L["kind"] != "pool":
            continue  # a valid convolution keeps the corner where it is
        sy, sx = syx(L)
        ox, oy = x % sx, y % sy
        x, y = x // sx, y // sy
        f = f * sy * sx + oy * sx + ox
        offs.append((ox, oy))
    return f, y, x, offs


def fragment_extents(layers, H, W):
    """Per layer (index 0 = input), the list of fragment sizes (s_y, s_x),
    fragment ids in list order."""
    frags = [(H, W)]
    out = [list(frags)]
    for L in layers:
        ky, kx = kyx(L)
        if L["kind"] == "pool":
            ty, tx = syx(L)
            nxt = []
            for (sy, sx) in frags:
                for oy in range(ty):
                    for ox in range(tx):
                        nxt.append((max(sy - oy - ky + ty, 0) // ty, max(sx - ox - kx + tx, 0) // tx))
            frags = nxt
        else:
            frags = [(max(sy - (ky - 1), 0), max(sx - (kx - 1), 0)) for (sy, sx) in frags]
        out.append(list(frags))
    return out


def n_fragments(layers):
    F = 1
    for L in layers:
        if L["kind"] == "pool":
            F *= syx(L)[0] * syx(L)[1]
    return F


def reassembly_index(layers, H, W):
    """[n_y, n_x, 3] int64 array of (f, y_f, x_f) for every output pixel."""
    h0, w0 = patch_hw(layers)
    ny, nx = H - h0 + 1, W - w0 + 1
    Y, X = np.meshgrid(np.arange(ny), np.arange(nx), indexing="ij")
    f, y, x, _ = track(layers, Y, X)
    return np.stack([f, y, x], axis=-1)


def fragment_table(layers, H, W):
    """Dict per final fragment id f present in the output:
       {"offsets": [(o_x, o_y) per pool], "base": (Y0, X0), "size": (h, w)}
    found by tracking every output pixel (a fragment with no valid output does
    not appear)."""
    h0, w0 = patch_hw(layers)
    ny, nx = H - h0 + 1, W - w0 + 1
    Y, X = np.meshgrid(np.arange(ny), np.arange(nx), indexing="ij")
    f, y, x, offs = track(layers, Y, X)
    table = {}
    for idx in np.ndindex(f.shape):
        fid = int(f[idx])
        e = table.get(fid)
        o = [(int(ox[idx]), int(oy[idx])) for (ox, oy) in offs]
        if e is None:
            e = {"offsets": o, "base": (int(Y[idx]), int(X[idx])), "ys": set(), "xs": set()}
            table[fid] = e
        if e["offsets"] != o:
            raise AssertionError("fragment %d reached with two offset chains" % fid)
        e["base"] = (min(e["base"][0], int(Y[idx])), min(e["base"][1], int(X[idx])))
        e["ys"].add(int(y[idx]))
        e["xs"].add(int(x[idx]))
    for e in table.values():
        e["size"] = (len(e.pop("ys")), len(e.pop("xs")))
    return table


def flops_patch(s, p_prev, p_l, w_l, k_l):
    """Section 3.1: s^2 * |P_{l-1}| * |P_l| * w_l^2 * k_l^2 * 2."""
    return s * s * p_prev * p_l * w_l * w_l * k_l * k_l * 2


def flops_image(s_x, s_y, p_prev, p_l, F_l, k_l):
    """Section 3.1: s_x * s_y * |P_{l-1}| * |P_l| * F_l * k_l^2 * 2 (all
    fragments taken to be s_x by s_y)."""
    return s_x * s_y * p_prev * p_l * F_l * k_l * k_l * 2


def algorithmic_flops(layers, B, H, W):
    """Per layer, 2 * c_in * k^2 * c_out times the number of output pixels
    summed over all fragments (pools: 0)."""
    ext = fragment_extents(layers, H, W)
    res = []
    for l, L in enumerate(layers):
        if L["kind"] == "pool":
            res.append(0)
            continue
        pix = sum(sy * sx for (sy, sx) in ext[l + 1])
        res.append(B * pix * 2 * L["c_in"] * kyx(L)[0] * kyx(L)[1] * L["c_out"])
    return res
