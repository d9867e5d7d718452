"""Pins of the fp64 CPU oracle against what the paper and mathematics fix.

Each test reaches the expected value by a route that does not reuse the
oracle's own algorithm: values the paper prints (tests/golden), closed forms,
independent constructions (tests/_independent.py), library primitives (torch
CPU float64 convolutions), finite differences and exact identities.
"""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
from tests import _independent as ind

RNG = np.random.default_rng(12345)

SIZES = [(1, 1), (1, 5), (6, 1), (2, 2), (5, 7), (8, 8), (9, 7), (13, 11), (16, 16), (7, 7)]


def _rand_params(C, k, L, rng=RNG, zero_levels=False):
    w0 = rng.uniform(-0.2, 0.2, (C, k, k))
    s0 = rng.uniform(0.5, 1.5, (C,))
    wl = [np.zeros((4 * C, k, k)) if zero_levels else rng.uniform(-0.2, 0.2, (4 * C, k, k)) for _ in range(L)]
    sl = [rng.uniform(0.05, 0.2, (4 * C,)) for _ in range(L)]
    return w0, s0, wl, sl


def _plane_params(wl, sl, c):
    return [wl[l][4 * c:4 * c + 4] for l in range(len(wl))], [sl[l][4 * c:4 * c + 4] for l in range(len(sl))]


# --------------------------------------------------------------------------
# Haar conventions pinned to the paper's printed matrix and sign table
# --------------------------------------------------------------------------

def test_haar_matrix_is_proposition_1(golden):
    rows = golden("haar_matrix.txt")
    Hp = np.array([[float(v) for v in r[1:]] for r in rows]) / 2.0
    assert [r[0] for r in rows] == ["LL", "LH", "HL", "HH"]
    # the oracle's analysis of each basis patch a, b, c, d gives one column of H
    M = np.zeros((4, 4))
    for pos in range(4):
        patch = np.zeros((2, 2))
        patch[pos // 2, pos % 2] = 1.0
        M[:, pos] = oracle.haar_analysis(patch)[:, 0, 0]
    np.testing.assert_array_equal(M, Hp)
    # Proposition 1: H^T = H and H^2 = I
    np.testing.assert_array_equal(M, M.T)
    np.testing.assert_allclose(M @ M, np.eye(4), atol=0, rtol=0)


def test_synthesis_sign_table(golden):
    rows = golden("haar_sign_table.txt")
    for ry, rx, *signs in rows:
        ry, rx = int(ry), int(rx)
        for q, sgn in zip((1, 2, 3), signs):
            coef = np.zeros((4, 1, 1))
            coef[q] = 1.0
            block = oracle.haar_synthesis(coef, 2, 2)
            assert block[ry, rx] == (0.5 if sgn == "+" else -0.5)
        coef = np.zeros((4, 1, 1))
        coef[0] = 1.0
        assert oracle.haar_synthesis(coef, 2, 2)[ry, rx] == 0.5


# --------------------------------------------------------------------------
# P1: perfect reconstruction and orthonormality (Proposition 1)
# --------------------------------------------------------------------------

@pytest.mark.parametrize("h,w", SIZES)
def test_perfect_reconstruction(h, w):
    X = RNG.standard_normal((h, w))
    Y = oracle.haar_analysis(X)
    assert Y.shape == (4, (h + 1) // 2, (w + 1) // 2)
    np.testing.assert_allclose(oracle.haar_synthesis(Y, h, w), X, rtol=0, atol=1e-14)
    # orthonormal: energy of the zero-padded block grid is preserved
    assert abs((Y ** 2).sum() - (X ** 2).sum()) <= 1e-12 * max(1.0, (X ** 2).sum())


@pytest.mark.parametrize("h,w", SIZES)
def test_analysis_synthesis_adjoint(h, w):
    X = RNG.standard_normal((h, w))
    Yr = RNG.standard_normal((4, (h + 1) // 2, (w + 1) // 2))
    lhs = (oracle.haar_analysis(X) * Yr).sum()
    rhs = (X * oracle.haar_synthesis(Yr, h, w)).sum()
    assert abs(lhs - rhs) <= 1e-12 * (abs(lhs) + 1)


# --------------------------------------------------------------------------
# P7: level-l coefficients of the zero-extended input
# --------------------------------------------------------------------------

@pytest.mark.parametrize("h,w,L", [(8, 8, 3), (9, 7, 2), (13, 11, 3), (7, 7, 5), (16, 16, 4), (5, 9, 3),
                                   (1, 1, 2), (56, 56, 3), (63, 95, 5)])
def test_pyramid_is_zero_extended_block_sums(h, w, L):
    x = RNG.standard_normal((h, w))
    got = oracle.plane_pyramid(x, L)
    want = ind.zero_extended_pyramid(x, L)
    for g, e in zip(got, want):
        assert g.shape == e.shape
        np.testing.assert_allclose(g, e, rtol=0, atol=1e-13)


# --------------------------------------------------------------------------
# P6: closed-form synthesis (Proposition 2) equals the cascade
# --------------------------------------------------------------------------

@pytest.mark.parametrize("h,w,L", [(8, 8, 1), (8, 8, 3), (9, 7, 2), (13, 11, 3), (7, 7, 5), (16, 16, 4),
                                   (5, 9, 3), (1, 1, 3), (63, 95, 5), (6, 6, 6)])
def test_closed_form_equals_cascade(h, w, L):
    levels = [RNG.standard_normal((4,) + ind.level_shape(h, w, l)) for l in range(1, L + 1)]
    cascade = oracle.cascade_synthesis(levels, h, w)
    np.testing.assert_allclose(oracle.closed_form_synthesis(levels, h, w), cascade, rtol=0, atol=1e-14)
    np.testing.assert_allclose(ind.closed_form(levels, h, w), cascade, rtol=0, atol=1e-14)


def test_bit_indexed_worked_example(golden):
    """A unit coefficient at level l reaches pixel (y, x) with weight 2^-l and the
    sign-table sign of bit (l-1) of y and x (Appendix A worked example)."""
    signs = {(int(r[0]), int(r[1])): r[2:] for r in golden("haar_sign_table.txt")}
    for level, shift, weight in golden("bit_indexed_example.txt"):
        level, shift, weight = int(level), int(shift), float(weight)
        H = W = 2 ** (level + 1)
        for q in range(4):
            levels = [np.zeros((4,) + ind.level_shape(H, W, l)) for l in range(1, level + 1)]
            levels[level - 1][q, 1, 0] = 1.0  # coefficient at coarse site (1, 0)
            R = oracle.cascade_synthesis(levels, H, W)
            for y in range(H):
                for x in range(W):
                    inside = (y >> level) == 1 and (x >> level) == 0
                    if not inside:
                        assert R[y, x] == 0.0
                        continue
                    by, bx = (y >> shift) & 1, (x >> shift) & 1
                    s = "+" if q == 0 else signs[(by, bx)][q - 1]
                    assert R[y, x] == (weight if s == "+" else -weight)


# --------------------------------------------------------------------------
# P4 / P5: library primitives (torch CPU float64)
# --------------------------------------------------------------------------

def _torch_conv_same(x, w):
    """Depthwise 'same' correlation with torch conv2d (groups = channels)."""
    C = x.shape[1]
    k = w.shape[-1]
    return F.conv2d(torch.from_numpy(x), torch.from_numpy(w).reshape(C, 1, k, k), padding=k // 2,
                    groups=C).numpy()


@pytest.mark.parametrize("B,C,H,W,k,L", [(2, 3, 9, 7, 5, 2), (1, 2, 8, 8, 3, 0), (2, 2, 5, 6, 7, 1)])
def test_zero_wavelet_weights_reduce_to_scaled_base_conv(B, C, H, W, k, L):
    x = RNG.standard_normal((B, C, H, W))
    w0, s0, wl, sl = _rand_params(C, k, L, zero_levels=True)
    got = oracle.forward(x, w0, s0, wl, sl)
    want = s0[None, :, None, None] * _torch_conv_same(x, w0)
    np.testing.assert_allclose(got, want, rtol=0, atol=1e-14)


def _torch_reference_chain(x, w0, s0, wl, sl):
    """Alg. 1 with the framework primitives the paper attributes to the reference
    implementation (Section 3.1): grouped stride-2 conv2d against fixed +-1/2
    filters, depthwise conv2d over the 4C coefficient channels, scale multiply,
    slice, add, cat, conv_transpose2d; base conv2d, multiply, add."""
    X = torch.from_numpy(x)
    B, C, H, W = X.shape
    k = w0.shape[-1]
    haar = torch.tensor([[1, 1, 1, 1], [1, 1, -1, -1], [1, -1, 1, -1], [1, -1, -1, 1]],
                        dtype=torch.float64).reshape(4, 1, 2, 2) * 0.5
    filt = haar.repeat(C, 1, 1, 1)  # [4C, 1, 2, 2], channel 4c+q
    carriers, shapes, zs = X, [], []
    for l in range(len(wl)):
        h, w = carriers.shape[-2:]
        shapes.append((h, w))
        padded = F.pad(carriers, (0, w % 2, 0, h % 2))
        Y = F.conv2d(padded, filt, stride=2, groups=C)  # [B, 4C, h', w']
        Z = F.conv2d(Y, torch.from_numpy(wl[l]).reshape(4 * C, 1, k, k), padding=k // 2, groups=4 * C)
        Z = Z * torch.from_numpy(sl[l]).reshape(1, 4 * C, 1, 1)
        zs.append(Z)
        carriers = Y[:, 0::4]
    R = None
    for l in reversed(range(len(wl))):
        Z = zs[l].clone()
        if R is not None:
            Z[:, 0::4] = Z[:, 0::4] + R
        S = F.conv_transpose2d(Z, filt, stride=2, groups=C)
        h, w = shapes[l]
        R = S[..., :h, :w]
    base = F.conv2d(X, torch.from_numpy(w0).reshape(C, 1, k, k), padding=k // 2, groups=C)
    out = base * torch.from_numpy(s0).reshape(1, C, 1, 1)
    if R is not None:
        out = out + R
    return out.numpy()


@pytest.mark.parametrize("B,C,H,W,k,L", [(2, 3, 16, 16, 5, 3), (1, 2, 9, 7, 3, 2), (2, 2, 13, 11, 5, 4),
                                         (1, 1, 7, 7, 5, 5), (2, 2, 32, 32, 5, 1), (1, 2, 5, 9, 7, 3)])
def test_matches_torch_primitive_chain(B, C, H, W, k, L):
    x = RNG.standard_normal((B, C, H, W))
    w0, s0, wl, sl = _rand_params(C, k, L)
    np.testing.assert_allclose(oracle.forward(x, w0, s0, wl, sl), _torch_reference_chain(x, w0, s0, wl, sl),
                               rtol=0, atol=1e-13)


def test_analysis_is_strided_conv_and_synthesis_is_transposed_conv():
    for h, w in [(8, 8), (9, 7), (5, 6)]:
        X = RNG.standard_normal((h, w))
        haar = torch.tensor([[1, 1, 1, 1], [1, 1, -1, -1], [1, -1, 1, -1], [1, -1, -1, 1]],
                            dtype=torch.float64).reshape(4, 1, 2, 2) * 0.5
        padded = F.pad(torch.from_numpy(X)[None, None], (0, w % 2, 0, h % 2))
        want = F.conv2d(padded, haar, stride=2)[0].numpy()
        np.testing.assert_allclose(oracle.haar_analysis(X), want, rtol=0, atol=1e-15)
        Y = RNG.standard_normal(want.shape)
        back = F.conv_transpose2d(torch.from_numpy(Y)[None], haar, stride=2)[0, 0, :h, :w].numpy()
        np.testing.assert_allclose(oracle.haar_synthesis(Y, h, w), back, rtol=0, atol=1e-15)


# --------------------------------------------------------------------------
# P2 / P3: identity kernels
# --------------------------------------------------------------------------

def _identity(k):
    e = np.zeros((k, k))
    e[k // 2, k // 2] = 1.0
    return e


@pytest.mark.parametrize("H,W,k,L", [(8, 8, 5, 1), (16, 16, 5, 3), (9, 7, 3, 2), (13, 11, 5, 4), (7, 7, 5, 5),
                                     (63, 95, 5, 5)])
def test_exact_reproduction_pattern(H, W, k, L):
    """Base zeroed; identity on LH/HL/HH at every level, identity on LL only at
    level L, zero LL kernels below it; unit scales: the branch returns x."""
    x = RNG.standard_normal((H, W))
    wl = np.zeros((L, 4, k, k))
    for l in range(L):
        for q in (1, 2, 3):
            wl[l, q] = _identity(k)
    wl[L - 1, 0] = _identity(k)
    y = oracle.plane_forward(x, np.zeros((k, k)), 1.0, wl, np.ones((L, 4)))
    np.testing.assert_allclose(y, x, rtol=0, atol=1e-13)


@pytest.mark.parametrize("H,W,k,L", [(8, 8, 5, 1), (16, 16, 5, 3), (9, 7, 3, 2), (13, 11, 5, 4), (7, 7, 5, 5)])
def test_all_identity_gives_block_means(H, W, k, L):
    """Identity kernels on every band of every level, unit scales, base zeroed:
    y = x + sum_{j=1}^{L-1} P_j x with P_j the 2^j block mean of the
    zero-extended input."""
    x = RNG.standard_normal((H, W))
    wl = np.stack([np.stack([_identity(k)] * 4)] * L)
    y = oracle.plane_forward(x, np.zeros((k, k)), 1.0, wl, np.ones((L, 4)))
    want = x + sum(ind.block_mean(x, j) for j in range(1, L))
    np.testing.assert_allclose(y, want, rtol=0, atol=1e-13)


# --------------------------------------------------------------------------
# Brute force: the dense operator built from the closed forms
# --------------------------------------------------------------------------

@pytest.mark.parametrize("H,W,k,L", [(8, 8, 5, 2), (9, 7, 3, 3), (5, 6, 5, 1), (7, 7, 5, 5), (4, 9, 3, 4)])
def test_dense_operator_from_closed_forms(H, W, k, L):
    x = RNG.standard_normal((H, W))
    dy = RNG.standard_normal((H, W))
    w0, s0, wl, sl = _rand_params(1, k, L)
    wlp, slp = _plane_params(wl, sl, 0)
    fn = lambda img: ind.operator_closed_form(img, w0[0], s0[0], wlp, slp)  # noqa: E731
    M = ind.dense_matrix(H, W, fn)
    y = oracle.plane_forward(x, w0[0], s0[0], np.stack(wlp) if L else [], np.stack(slp) if L else [])
    np.testing.assert_allclose(y, (M @ x.ravel()).reshape(H, W), rtol=0, atol=1e-13)
    dx = oracle.plane_backward(x, dy, w0[0], s0[0], np.stack(wlp) if L else [], np.stack(slp) if L else [])[0]
    np.testing.assert_allclose(dx, (M.T @ dy.ravel()).reshape(H, W), rtol=0, atol=1e-13)


# --------------------------------------------------------------------------
# P8 / P9: adjoint identities of the backward pass
# --------------------------------------------------------------------------

@pytest.mark.parametrize("B,C,H,W,k,L", [(2, 3, 16, 16, 5, 3), (1, 2, 13, 11, 3, 4), (2, 2, 7, 7, 5, 5)])
def test_dot_product_adjoint(B, C, H, W, k, L):
    x = RNG.standard_normal((B, C, H, W))
    dy = RNG.standard_normal((B, C, H, W))
    w0, s0, wl, sl = _rand_params(C, k, L)
    y = oracle.forward(x, w0, s0, wl, sl)
    g = oracle.backward(x, dy, w0, s0, wl, sl)
    lhs, rhs = (y * dy).sum(), (x * g["dx"]).sum()
    assert abs(lhs - rhs) <= 1e-12 * max(1.0, abs(lhs))


@pytest.mark.parametrize("B,C,H,W,k,L", [(2, 3, 16, 16, 5, 3), (1, 2, 13, 11, 3, 4), (2, 2, 9, 7, 7, 2)])
def test_dx_is_forward_with_rotated_kernels(B, C, H, W, k, L):
    x = RNG.standard_normal((B, C, H, W))
    dy = RNG.standard_normal((B, C, H, W))
    w0, s0, wl, sl = _rand_params(C, k, L)
    dx = oracle.backward(x, dy, w0, s0, wl, sl)["dx"]
    rot = lambda a: a[..., ::-1, ::-1].copy()  # noqa: E731
    want = oracle.forward(dy, rot(w0), s0, [rot(w) for w in wl], sl)
    np.testing.assert_allclose(dx, want, rtol=0, atol=1e-13)


# --------------------------------------------------------------------------
# P10: central finite differences for every gradient on tiny inputs
# --------------------------------------------------------------------------

@pytest.mark.parametrize("H,W,k,L", [(5, 5, 3, 1), (8, 8, 5, 2), (9, 7, 3, 3), (5, 9, 5, 2)])
def test_finite_differences(H, W, k, L):
    B, C = 2, 2
    x = RNG.standard_normal((B, C, H, W))
    dy = RNG.standard_normal((B, C, H, W))
    w0, s0, wl, sl = _rand_params(C, k, L)
    g = oracle.backward(x, dy, w0, s0, wl, sl)
    h = 1e-3

    def loss(x_, w0_, s0_, wl_, sl_):
        return float((oracle.forward(x_, w0_, s0_, wl_, sl_) * dy).sum())

    def fd(arr, idx, call):
        a0 = arr[idx]
        arr[idx] = a0 + h
        up = call()
        arr[idx] = a0 - h
        dn = call()
        arr[idx] = a0
        return (up - dn) / (2 * h)

    call = lambda: loss(x, w0, s0, wl, sl)  # noqa: E731
    scale = max(1.0, np.abs(g["dx"]).max())
    for idx in [(0, 0, 0, 0), (1, 1, H - 1, W - 1), (0, 1, H // 2, W // 3), (1, 0, 1, W - 2)]:
        assert abs(fd(x, idx, call) - g["dx"][idx]) <= 1e-7 * scale
    for idx in np.ndindex(w0.shape):
        assert abs(fd(w0, idx, call) - g["d_base_w"][idx]) <= 1e-7 * max(1.0, abs(g["d_base_w"][idx]))
    for c in range(C):
        assert abs(fd(s0, (c,), call) - g["d_base_scale"][c]) <= 1e-7 * max(1.0, abs(g["d_base_scale"][c]))
    for l in range(L):
        for idx in np.ndindex(wl[l].shape):
            ref = g["d_level_w"][l][idx]
            assert abs(fd(wl[l], idx, call) - ref) <= 1e-7 * max(1.0, abs(ref))
        for idx in np.ndindex(sl[l].shape):
            ref = g["d_level_scale"][l][idx]
            assert abs(fd(sl[l], idx, call) - ref) <= 1e-7 * max(1.0, abs(ref))


# --------------------------------------------------------------------------
# P11: homogeneity identities behind eq. (foldgrad)
# --------------------------------------------------------------------------

@pytest.mark.parametrize("B,C,H,W,k,L", [(4, 8, 32, 32, 5, 3), (2, 4, 28, 28, 5, 5), (2, 3, 15, 21, 3, 2)])
def test_homogeneity_identities(B, C, H, W, k, L):
    """Each branch is linear in its kernel and in its scale, so
    sum(dW * W) = sum(s * ds) = <dy, branch output> for the base path and for
    every level (Euler's identity; the fold of eq. (foldgrad) relies on it)."""
    rng = np.random.default_rng(7)
    x = rng.standard_normal((B, C, H, W))
    dy = rng.standard_normal((B, C, H, W))
    w0, s0, wl, sl = _rand_params(C, k, L, rng)
    g = oracle.backward(x, dy, w0, s0, wl, sl)
    zero = [np.zeros_like(w) for w in wl]
    base = oracle.forward(x, w0, s0, zero, sl)
    ref = (dy * base).sum()
    assert abs((g["d_base_w"] * w0).sum() - ref) <= 1e-11 * abs(ref)
    assert abs((g["d_base_scale"] * s0).sum() - ref) <= 1e-11 * abs(ref)
    for l in range(L):
        only = [wl[m] if m == l else zero[m] for m in range(L)]
        branch = oracle.forward(x, np.zeros_like(w0), s0, only, sl)
        ref = (dy * branch).sum()
        assert abs((g["d_level_w"][l] * wl[l]).sum() - ref) <= 1e-11 * abs(ref)
        assert abs((g["d_level_scale"][l] * sl[l]).sum() - ref) <= 1e-11 * abs(ref)


def test_batch_sum_order_and_plane_independence():
    B, C, H, W, k, L = 3, 2, 9, 7, 5, 2
    x = RNG.standard_normal((B, C, H, W))
    dy = RNG.standard_normal((B, C, H, W))
    w0, s0, wl, sl = _rand_params(C, k, L)
    y = oracle.forward(x, w0, s0, wl, sl)
    g = oracle.backward(x, dy, w0, s0, wl, sl)
    acc_w0 = np.zeros_like(w0)
    for b in range(B):
        for c in range(C):
            wlp, slp = _plane_params(wl, sl, c)
            np.testing.assert_array_equal(y[b, c], oracle.plane_forward(x[b, c], w0[c], s0[c], np.stack(wlp),
                                                                        np.stack(slp)))
            dxp, dw0p, *_ = oracle.plane_backward(x[b, c], dy[b, c], w0[c], s0[c], np.stack(wlp), np.stack(slp))
            np.testing.assert_array_equal(g["dx"][b, c], dxp)
            acc_w0[c] += dw0p
    np.testing.assert_array_equal(g["d_base_w"], acc_w0)


# --------------------------------------------------------------------------
# P12: the base bias of Algorithm 1 (y = s0 (x * W0 + b) + R) and its
# gradients, eq. (fold) / eq. (foldgrad): db = s0 * sum(dy),
# ds0 = <dW~, W0> + db~ * b with db~ = sum(dy)
# --------------------------------------------------------------------------

@pytest.mark.parametrize("B,C,H,W,k,L", [(2, 3, 9, 7, 5, 2), (1, 2, 8, 8, 3, 0), (2, 2, 5, 6, 7, 1)])
def test_bias_matches_torch_conv2d_bias(B, C, H, W, k, L):
    """Zero wavelet weights: y = s0 * conv2d(x, W0, bias=b), torch float64."""
    x = RNG.standard_normal((B, C, H, W))
    w0, s0, wl, sl = _rand_params(C, k, L, zero_levels=True)
    b = RNG.uniform(-1, 1, (C,))
    got = oracle.forward(x, w0, s0, wl, sl, base_bias=b)
    want = F.conv2d(torch.from_numpy(x), torch.from_numpy(w0).reshape(C, 1, k, k), bias=torch.from_numpy(b),
                    padding=k // 2, groups=C).numpy() * s0[None, :, None, None]
    np.testing.assert_allclose(got, want, rtol=0, atol=1e-14)


def test_bias_only_closed_form():
    """All kernels zero: y = s0 * b everywhere; db = s0 * sum(dy), ds0 = b * sum(dy),
    and dx = 0."""
    B, C, H, W, k, L = 3, 4, 7, 9, 5, 3
    rng = np.random.default_rng(3)
    x = rng.standard_normal((B, C, H, W))
    dy = rng.standard_normal((B, C, H, W))
    s0 = rng.uniform(0.5, 1.5, (C,))
    b = rng.uniform(-1, 1, (C,))
    wl = [np.zeros((4 * C, k, k)) for _ in range(L)]
    sl = [rng.uniform(0.05, 0.2, (4 * C,)) for _ in range(L)]
    y = oracle.forward(x, np.zeros((C, k, k)), s0, wl, sl, base_bias=b)
    np.testing.assert_array_equal(y, np.broadcast_to((s0 * b)[None, :, None, None], y.shape))
    g = oracle.backward(x, dy, np.zeros((C, k, k)), s0, wl, sl, base_bias=b)
    sdy = dy.sum(axis=(0, 2, 3))
    np.testing.assert_allclose(g["d_base_bias"], s0 * sdy, rtol=1e-13, atol=0)
    np.testing.assert_allclose(g["d_base_scale"], b * sdy, rtol=1e-13, atol=0)
    assert not np.any(g["dx"])


@pytest.mark.parametrize("H,W,k,L", [(5, 5, 3, 1), (8, 8, 5, 2), (9, 7, 3, 3)])
def test_bias_finite_differences(H, W, k, L):
    B, C = 2, 2
    x = RNG.standard_normal((B, C, H, W))
    dy = RNG.standard_normal((B, C, H, W))
    w0, s0, wl, sl = _rand_params(C, k, L)
    b = RNG.uniform(-1, 1, (C,))
    g = oracle.backward(x, dy, w0, s0, wl, sl, base_bias=b)
    h = 1e-3

    def loss():
        return float((oracle.forward(x, w0, s0, wl, sl, base_bias=b) * dy).sum())

    def fd(arr, idx):
        a0 = arr[idx]
        arr[idx] = a0 + h
        up = loss()
        arr[idx] = a0 - h
        dn = loss()
        arr[idx] = a0
        return (up - dn) / (2 * h)

    for c in range(C):
        assert abs(fd(b, (c,)) - g["d_base_bias"][c]) <= 1e-7 * max(1.0, abs(g["d_base_bias"][c]))
        assert abs(fd(s0, (c,)) - g["d_base_scale"][c]) <= 1e-7 * max(1.0, abs(g["d_base_scale"][c]))
    # dx and the kernel gradients do not depend on the bias
    g0 = oracle.backward(x, dy, w0, s0, wl, sl)
    np.testing.assert_array_equal(g["dx"], g0["dx"])
    np.testing.assert_array_equal(g["d_base_w"], g0["d_base_w"])


def test_bias_homogeneity():
    """The base branch s0 (x * W0 + b) is linear in (W0, b) jointly and in s0:
    sum(dW0 W0) + sum(db b) = sum(ds0 s0) = <dy, base branch>."""
    B, C, H, W, k, L = 2, 5, 16, 12, 5, 2
    rng = np.random.default_rng(11)
    x = rng.standard_normal((B, C, H, W))
    dy = rng.standard_normal((B, C, H, W))
    w0, s0, wl, sl = _rand_params(C, k, L, rng)
    b = rng.uniform(-1, 1, (C,))
    g = oracle.backward(x, dy, w0, s0, wl, sl, base_bias=b)
    zero = [np.zeros_like(w) for w in wl]
    ref = (dy * oracle.forward(x, w0, s0, zero, sl, base_bias=b)).sum()
    assert abs((g["d_base_w"] * w0).sum() + (g["d_base_bias"] * b).sum() - ref) <= 1e-11 * abs(ref)
    assert abs((g["d_base_scale"] * s0).sum() - ref) <= 1e-11 * abs(ref)
