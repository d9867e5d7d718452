"""Independent numpy constructions used to pin the oracle.

None of these reuse the oracle's code or its algorithm (the Alg. 1 cascade
with per-level pad/crop): they follow other statements of the paper, or facts
derived from it, written out directly.
"""
import numpy as np
from scipy.signal import correlate2d


def level_shape(H, W, l):
    for _ in range(l):
        H, W = (H + 1) // 2, (W + 1) // 2
    return H, W


def zero_extended_pyramid(x, L):
    """Level-l Haar coefficients as 2^-l times signed quadrant sums of the
    2^l x 2^l block of the zero-extended input (each level's LL is 2^-l times
    the block sum; LH top minus bottom; HL left minus right; HH the diagonal
    difference)."""
    H, W = x.shape
    out = []
    for l in range(1, L + 1):
        h, w = level_shape(H, W, l)
        s = 2 ** l
        ext = np.zeros((h * s, w * s))
        ext[:H, :W] = x
        blk = ext.reshape(h, s, w, s).transpose(0, 2, 1, 3)  # [h, w, s, s]
        half = s // 2
        tl = blk[:, :, :half, :half].sum(axis=(2, 3))
        tr = blk[:, :, :half, half:].sum(axis=(2, 3))
        bl = blk[:, :, half:, :half].sum(axis=(2, 3))
        br = blk[:, :, half:, half:].sum(axis=(2, 3))
        sc = 2.0 ** (-l)
        out.append(np.stack([sc * (tl + tr + bl + br), sc * (tl + tr - bl - br),
                             sc * (tl - tr + bl - br), sc * (tl - tr - bl + br)]))
    return out


def closed_form(levels, H, W):
    """Proposition 2 evaluated for every pixel at once."""
    yy, xx = np.meshgrid(np.arange(H), np.arange(W), indexing="ij")
    R = np.zeros((H, W))
    for l, c in enumerate(levels, start=1):
        j, i = yy >> l, xx >> l
        sy = np.where((yy >> (l - 1)) & 1, -1.0, 1.0)
        sx = np.where((xx >> (l - 1)) & 1, -1.0, 1.0)
        R += 2.0 ** (-l) * (c[0][j, i] + sy * c[1][j, i] + sx * c[2][j, i] + sy * sx * c[3][j, i])
    return R


def corr_same(u, wk):
    """Zero-padded 'same' cross-correlation via scipy (odd kernel)."""
    return correlate2d(u, wk, mode="same", boundary="fill", fillvalue=0.0)


def operator_closed_form(x, w0, s0, wl, sl):
    """y = s0 (x * W0) + sum_l S_l( s_l (T_l x * W_l) ), with T_l from the
    zero-extension formula and S_l the bit-indexed closed form."""
    H, W = x.shape
    L = len(wl)
    pyr = zero_extended_pyramid(x, L)
    z = [np.stack([sl[l][q] * corr_same(pyr[l][q], wl[l][q]) for q in range(4)]) for l in range(L)]
    return s0 * corr_same(x, w0) + (closed_form(z, H, W) if L else 0.0)


def dense_matrix(H, W, fn):
    """Matrix of a linear map on H x W images, built column by column."""
    n = H * W
    M = np.zeros((n, n))
    for e in range(n):
        b = np.zeros(n)
        b[e] = 1.0
        M[:, e] = fn(b.reshape(H, W)).ravel()
    return M


def block_mean(x, j):
    """P_j: mean over the 2^j x 2^j block of the zero-extended input, cropped."""
    H, W = x.shape
    s = 2 ** j
    h, w = -(-H // s), -(-W // s)
    ext = np.zeros((h * s, w * s))
    ext[:H, :W] = x
    m = ext.reshape(h, s, w, s).mean(axis=(1, 3))
    return np.repeat(np.repeat(m, s, axis=0), s, axis=1)[:H, :W]
