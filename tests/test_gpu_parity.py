"""GPU parity: the fused HIP path, called through the C ABI, against the float64
oracle on the same seeded (and storage-rounded) inputs.

Tolerances (max abs error over max abs reference, per tensor): 1e-5 for fp32,
2e-2 for bf16 / fp16 storage (fp32 accumulation in both cases).
"""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

import oracle  # noqa: E402
from tests._gpu import TOL, channel_slice, rel_err, setup, to_np  # noqa: E402

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():
    pytest.skip("needs a GPU", allow_module_level=True)


def check_forward(B, C, H, W, k, L, dtype, seed=0):
    inp, dev = setup(B, C, H, W, k, L, dtype, seed)
    y = to_np(dev.forward())
    ref = oracle.forward(inp.x, inp.base_w, inp.base_scale, inp.level_w, inp.level_scale)
    e = rel_err(y, ref)
    assert e < TOL[dtype], f"forward rel err {e:.3e}"
    return e


def check_backward(B, C, H, W, k, L, dtype, seed=0, need_dx=True):
    inp, dev = setup(B, C, H, W, k, L, dtype, seed)
    dx, dbw, dbs, dlw, dls = dev.backward(need_dx=need_dx)
    ref = oracle.backward(inp.x, inp.dy, inp.base_w, inp.base_scale, inp.level_w, inp.level_scale)
    errs = {"d_base_w": rel_err(to_np(dbw), ref["d_base_w"]),
            "d_base_scale": rel_err(to_np(dbs), ref["d_base_scale"])}
    if need_dx:
        errs["dx"] = rel_err(to_np(dx), ref["dx"])
    for l in range(L):
        errs[f"d_level_w{l + 1}"] = rel_err(to_np(dlw[l]), ref["d_level_w"][l])
        errs[f"d_level_scale{l + 1}"] = rel_err(to_np(dls[l]), ref["d_level_scale"][l])
    tol = TOL[dtype]
    bad = {k_: v for k_, v in errs.items() if not v < tol}
    assert not bad, f"backward rel errs over {tol}: {bad}"
    return errs


# shapes small enough for the oracle to check every element, spanning several
# tiles, ragged tails, odd and 1-pixel sizes, every kernel size and L = 0..8
SMALL = [
    (2, 16, 32, 32, 5, 1, "f32"),   # the small forward workload
    (2, 3, 13, 11, 5, 3, "f32"),
    (1, 2, 7, 7, 5, 5, "f32"),      # grids reaching 1 x 1
    (2, 2, 1, 1, 3, 2, "f32"),
    (1, 1, 1, 9, 5, 2, "f32"),
    (3, 2, 9, 1, 3, 1, "f32"),
    (2, 4, 28, 28, 5, 4, "f32"),
    (1, 2, 63, 95, 5, 5, "f32"),
    (2, 2, 56, 56, 5, 3, "f32"),
    (2, 3, 17, 23, 1, 2, "f32"),
    (2, 3, 17, 23, 3, 3, "f32"),
    (2, 3, 17, 23, 7, 2, "f32"),
    (2, 2, 20, 20, 5, 0, "f32"),
    (1, 2, 40, 36, 5, 8, "f32"),
    (5, 3, 14, 14, 5, 2, "f32"),    # several planes resident per workgroup
    (3, 2, 40, 40, 5, 3, "f32"),    # levels >= 3 share level 1's round, 2 planes + a ragged batch
    (3, 2, 40, 40, 3, 5, "f32"),
    (9, 2, 7, 7, 3, 3, "f32"),
    (2, 4, 28, 28, 5, 3, "bf16"),
    (2, 3, 13, 11, 5, 2, "bf16"),
    (2, 4, 28, 28, 5, 3, "f16"),
    (1, 2, 63, 95, 3, 4, "f16"),
]


@pytest.mark.parametrize("B,C,H,W,k,L,dtype", SMALL)
def test_forward_small(B, C, H, W, k, L, dtype):
    check_forward(B, C, H, W, k, L, dtype)


@pytest.mark.parametrize("B,C,H,W,k,L,dtype", SMALL)
def test_backward_small(B, C, H, W, k, L, dtype):
    check_backward(B, C, H, W, k, L, dtype)


# The base bias of Algorithm 1 (folded as s0 * b0, eq. fold) through every
# execution mode: fused backward, gradient pass, tiny planes, split levels and
# large-plane regions; d_base_scale gains b0 * sum(dy) and d_base_bias is
# s0 * sum(dy) (eq. foldgrad).
BIAS = [
    (2, 3, 13, 11, 5, 3, "f32"),      # fused backward
    (2, 4, 28, 28, 5, 3, "f32"),      # gradient pass
    (70, 3, 7, 6, 5, 4, "f32"),       # tiny planes
    (2, 2, 56, 56, 5, 5, "f32"),      # split levels
    (1, 2, 130, 126, 5, 3, "f32"),    # region tiles
    (2, 4, 28, 28, 3, 2, "bf16"),
    (10, 3, 14, 14, 5, 2, "f32"),     # mixed forward rounds
]


@pytest.mark.parametrize("B,C,H,W,k,L,dtype", BIAS)
def test_bias_forward_backward(B, C, H, W, k, L, dtype):
    from paper_2608_10805_amd import binding
    from paper_2608_10805_amd.inputs import make_bias

    inp, dev = setup(B, C, H, W, k, L, dtype)
    b = make_bias(C)
    bt = torch.from_numpy(b).to("cuda:0")
    tol = TOL[dtype]
    y = binding.forward(dev.x, dev.bw, dev.bs, dev.lw, dev.ls, bias=bt)
    torch.cuda.synchronize()
    ref_y = oracle.forward(inp.x, inp.base_w, inp.base_scale, inp.level_w, inp.level_scale, base_bias=b)
    assert rel_err(to_np(y), ref_y) < tol
    dx, dbw, dbs, dlw, dls, dbb = binding.backward(dev.x, dev.dy, dev.bw, dev.bs, dev.lw, dev.ls, bias=bt,
                                                   need_dbias=True)
    torch.cuda.synchronize()
    ref = oracle.backward(inp.x, inp.dy, inp.base_w, inp.base_scale, inp.level_w, inp.level_scale, base_bias=b)
    errs = {"dx": rel_err(to_np(dx), ref["dx"]), "d_base_w": rel_err(to_np(dbw), ref["d_base_w"]),
            "d_base_scale": rel_err(to_np(dbs), ref["d_base_scale"]),
            "d_base_bias": rel_err(to_np(dbb), ref["d_base_bias"])}
    for l in range(L):
        errs[f"d_level_w{l + 1}"] = rel_err(to_np(dlw[l]), ref["d_level_w"][l])
        errs[f"d_level_scale{l + 1}"] = rel_err(to_np(dls[l]), ref["d_level_scale"][l])
    bad = {k_: v for k_, v in errs.items() if not v < tol}
    assert not bad, f"rel errs over {tol}: {bad}"


# wtconv_backward runs the finalize of the gradient route's kernel gradients
# (levels 0..Lf) in extra workgroups at the end of the dx launch; the
# two-phase calls (wtconv_backward_partials, then wtconv_backward_finalize)
# run it as a launch of its own. Same sums in the same order: bit-identical
# results, and the combined call within tolerance of the oracle.
TWO_PHASE = [
    (2, 8, 56, 56, 5, 3, "f32"),      # gradient pass, resident dx
    (2, 4, 28, 28, 5, 4, "f32"),      # coarse gradient route: dx with the coarse carry
    (3, 4, 12, 12, 5, 3, "f32"),      # the same with a mixed-round dx
    (10, 3, 14, 14, 5, 2, "bf16"),    # mixed-round dx
    (2, 2, 56, 56, 5, 5, "f32"),      # split dx
    (2, 2, 112, 112, 5, 3, "f32"),    # region dx
    (4, 8, 8, 8, 5, 2, "f32"),        # tiny planes (no gradient pass)
    (2, 3, 13, 11, 5, 3, "f16"),      # fused backward (no gradient pass)
]


@pytest.mark.parametrize("B,C,H,W,k,L,dtype", TWO_PHASE)
def test_combined_backward_matches_two_phase(B, C, H, W, k, L, dtype):
    from paper_2608_10805_amd import binding

    inp, dev = setup(B, C, H, W, k, L, dtype)
    bk = binding.Backward(dev.x, dev.bw, dev.bs, dev.lw, dev.ls, need_dx=True)
    outs = lambda: [bk.dx, bk.dbw, bk.dbs] + bk.dlw + bk.dls  # noqa: E731
    got = []
    for combined in (True, False):
        for t in outs():
            t.fill_(float("nan"))  # a skipped write shows
        if combined:
            bk.run(dev.x, dev.dy)
        else:
            bk.partials(dev.x, dev.dy)
            bk.finalize()
        torch.cuda.synchronize()
        got.append([t.clone() for t in outs()])
    names = ["dx", "d_base_w", "d_base_scale"] + [f"d_level_w{l + 1}" for l in range(L)] + \
        [f"d_level_scale{l + 1}" for l in range(L)]
    diff = [n for n, a, b in zip(names, *got) if not torch.equal(a, b)]
    assert not diff, f"combined and two-phase backward differ in {diff}"
    ref = oracle.backward(inp.x, inp.dy, inp.base_w, inp.base_scale, inp.level_w, inp.level_scale)
    want = [ref["dx"], ref["d_base_w"], ref["d_base_scale"]] + list(ref["d_level_w"]) + list(ref["d_level_scale"])
    errs = {n: rel_err(to_np(a), w) for n, a, w in zip(names, got[0], want)}
    bad = {n: v for n, v in errs.items() if not v < TOL[dtype]}
    assert not bad, f"rel errs over {TOL[dtype]}: {bad}"


def test_bias_autograd_module():
    from paper_2608_10805_amd.autograd import WTConv2d

    torch.manual_seed(1)
    m = WTConv2d(5, kernel_size=5, levels=2, bias=True, device="cuda:0")
    with torch.no_grad():
        m.base_bias.uniform_(-0.5, 0.5)
    x = torch.randn(2, 5, 24, 20, device="cuda:0", requires_grad=True)
    y = m(x)
    g = torch.randn_like(y)
    y.backward(g)
    c64 = lambda t: t.detach().cpu().double().numpy()  # noqa: E731
    lw = [c64(p) for p in m.level_w]
    ls = [c64(p) for p in m.level_scale]
    args = (c64(x), c64(m.base_w), c64(m.base_scale), lw, ls)
    assert rel_err(to_np(y), oracle.forward(*args, base_bias=c64(m.base_bias))) < 1e-5
    ref = oracle.backward(args[0], c64(g), *args[1:], base_bias=c64(m.base_bias))
    assert rel_err(to_np(x.grad), ref["dx"]) < 1e-5
    assert rel_err(to_np(m.base_scale.grad), ref["d_base_scale"]) < 1e-5
    assert rel_err(to_np(m.base_bias.grad), ref["d_base_bias"]) < 1e-5


# dx alone (the forward pass on dy with rotated kernels) in every execution
# mode of the forward: resident, tiny, split, region, 16-bit storage.
DATA = [
    (2, 4, 28, 28, 5, 3, "f32"),
    (70, 3, 7, 6, 5, 4, "f32"),
    (2, 2, 56, 56, 5, 5, "f32"),
    (1, 2, 130, 126, 5, 3, "f32"),
    (2, 3, 17, 23, 7, 2, "bf16"),
    (3, 2, 9, 1, 3, 1, "f16"),
]


@pytest.mark.parametrize("B,C,H,W,k,L,dtype", DATA)
def test_backward_data(B, C, H, W, k, L, dtype):
    from paper_2608_10805_amd import binding

    inp, dev = setup(B, C, H, W, k, L, dtype)
    dx = binding.backward_data(dev.dy, dev.bw, dev.bs, dev.lw, dev.ls)
    torch.cuda.synchronize()
    ref = oracle.backward(inp.x, inp.dy, inp.base_w, inp.base_scale, inp.level_w, inp.level_scale)
    e = rel_err(to_np(dx), ref["dx"])
    assert e < TOL[dtype], f"dx rel err {e:.3e}"


# Planes of at most 16 x 16 take the forward with mixed task rounds (output
# tiles and every (level, band) tile packed into rounds of 256 lanes): several
# resident planes with a partial last batch, odd sizes, k = 1..7, levels down
# to 1 x 1 grids, 16-bit storage; y, and dx (the same kernel on dy with
# rotated taps), against the oracle element by element.
MIXED = [
    (9, 6, 14, 14, 5, 1, "f32"),
    (11, 7, 14, 14, 5, 3, "f32"),
    (13, 5, 14, 14, 5, 2, "bf16"),
    (17, 3, 13, 15, 5, 1, "f32"),
    (5, 4, 16, 16, 7, 2, "f16"),
    (33, 2, 12, 12, 3, 2, "f32"),
    (6, 3, 9, 11, 1, 4, "f32"),
    (20, 2, 16, 10, 5, 8, "f32"),
]


@pytest.mark.parametrize("B,C,H,W,k,L,dtype", MIXED)
def test_mixed_rounds_forward_and_dx(B, C, H, W, k, L, dtype):
    from paper_2608_10805_amd import binding

    check_forward(B, C, H, W, k, L, dtype)
    inp, dev = setup(B, C, H, W, k, L, dtype)
    dx = binding.backward_data(dev.dy, dev.bw, dev.bs, dev.lw, dev.ls)
    torch.cuda.synchronize()
    ref = oracle.backward(inp.x, inp.dy, inp.base_w, inp.base_scale, inp.level_w, inp.level_scale)
    e = rel_err(to_np(dx), ref["dx"])
    assert e < TOL[dtype], f"dx rel err {e:.3e}"


def test_backward_without_dx_matches():
    check_backward(3, 4, 21, 19, 5, 3, "f32", need_dx=False)


# Planes above 16 x 16 with L >= 2 take the gradient pass (dx as the forward
# pass on dy with rotated kernels, kernel gradients from the dedicated pass).
# One resident plane per batch with several batches per workgroup stores the
# dy level-1 pyramid over the x plane and re-zeroes its halo ring between
# batches; the cases also cover odd sizes whose tiles do not divide the grid,
# k = 3 and 7, 16-bit storage and deep levels down to 1 x 1 grids.
GRAD = [
    (3, 512, 48, 48, 5, 3, "f32"),
    (3, 300, 50, 46, 3, 2, "f32"),
    (3, 400, 52, 52, 7, 4, "bf16"),
    (2, 3, 45, 61, 5, 6, "f32"),
    (6, 5, 30, 18, 5, 2, "f16"),
    (7, 3, 19, 19, 7, 2, "f32"),  # level-1 tiles over three rounds, 6 resident planes and a ragged batch
    (4, 6, 33, 29, 5, 1, "bf16"),  # one level
    (2, 3, 63, 95, 5, 3, "f32"),  # more 4x4 blocks than threads: two block rounds per plane
    (3, 260, 65, 61, 5, 2, "f32"),  # two block rounds, three planes per workgroup in turn
    (2, 3, 65, 61, 3, 2, "bf16"),
    (1, 2, 70, 66, 7, 1, "f16"),
    (1, 2, 97, 90, 3, 2, "bf16"),  # three block rounds
    (1, 3, 112, 112, 5, 3, "f32"),  # four block rounds
    (5, 3, 14, 14, 5, 2, "f32"),  # level 1 at most 8 x 8, L <= 2: several resident planes
    (3, 4, 11, 13, 3, 1, "bf16"),
    (2, 3, 16, 16, 7, 2, "f16"),
    (1, 2, 63, 95, 5, 4, "f32"),  # dy levels 3-4 stored past dy level 1 over the x plane
    (2, 3, 63, 95, 3, 5, "bf16"),
    # small planes with deep levels: the split at m = 1 (k = 7, and k = 5 on
    # planes of at most 3 x 3 pixel blocks)
    (3, 4, 12, 12, 5, 3, "f32"),
    (2, 3, 14, 14, 7, 3, "f32"),
    (2, 2, 16, 16, 7, 5, "bf16"),
    (5, 3, 11, 10, 5, 4, "f32"),
]


@pytest.mark.parametrize("B,C,H,W,k,L,dtype", GRAD)
def test_grad_pass_backward(B, C, H, W, k, L, dtype):
    check_backward(B, C, H, W, k, L, dtype)


def test_grad_pass_backward_without_dx():
    check_backward(3, 512, 48, 48, 5, 3, "f32", need_dx=False)


def _sample_planes(B, C, n, rng):
    picks = {(0, 0), (B - 1, C - 1)}
    while len(picks) < n:
        picks.add((int(rng.integers(B)), int(rng.integers(C))))
    return sorted(picks)


def check_full_size(B, C, H, W, k, L, dtype, backward, n_planes=12, n_channels=3, seed=0):
    """Full-size run in the benchmark's launch configuration; the oracle checks
    sampled planes of y / dx and all parameter gradients of sampled channels."""
    inp, dev = setup(B, C, H, W, k, L, dtype, seed)
    rng = np.random.default_rng(1)
    planes = _sample_planes(B, C, n_planes, rng)
    tol = TOL[dtype]
    y = dev.forward()
    for b, c in planes:
        wl = np.stack([w[4 * c:4 * c + 4] for w in inp.level_w]) if L else []
        sl = np.stack([s[4 * c:4 * c + 4] for s in inp.level_scale]) if L else []
        ref = oracle.plane_forward(inp.x[b, c], inp.base_w[c], inp.base_scale[c], wl, sl)
        e = rel_err(to_np(y[b, c]), ref)
        assert e < tol, f"y plane {(b, c)} rel err {e:.3e}"
    del y
    if not backward:
        return
    dx, dbw, dbs, dlw, dls = dev.backward()
    for b, c in planes:
        wl = np.stack([w[4 * c:4 * c + 4] for w in inp.level_w]) if L else []
        sl = np.stack([s[4 * c:4 * c + 4] for s in inp.level_scale]) if L else []
        ref = oracle.plane_backward(inp.x[b, c], inp.dy[b, c], inp.base_w[c], inp.base_scale[c], wl, sl)[0]
        e = rel_err(to_np(dx[b, c]), ref)
        assert e < tol, f"dx plane {(b, c)} rel err {e:.3e}"
    cs = sorted({0, C - 1} | {int(v) for v in rng.integers(0, C, n_channels)})
    xs, dys, bws, bss, lws, lss = channel_slice(inp, cs)
    ref = oracle.backward(xs, dys, bws, bss, lws, lss)
    idx = np.asarray(cs)
    sub4 = lambda t: to_np(t).reshape(C, 4, *t.shape[1:])[idx].reshape(-1, *t.shape[1:])  # noqa: E731
    errs = {"d_base_w": rel_err(to_np(dbw)[idx], ref["d_base_w"]),
            "d_base_scale": rel_err(to_np(dbs)[idx], ref["d_base_scale"])}
    for l in range(L):
        errs[f"d_level_w{l + 1}"] = rel_err(sub4(dlw[l]), ref["d_level_w"][l])
        errs[f"d_level_scale{l + 1}"] = rel_err(sub4(dls[l]), ref["d_level_scale"][l])
    bad = {k_: v for k_, v in errs.items() if not v < tol}
    assert not bad, f"full-size gradient rel errs over {tol}: {bad}"


def test_convnext_stage1_forward_full():
    """B=64 C=96 56x56, k=5, L=3, fp32 (forward workload)."""
    check_full_size(64, 96, 56, 56, 5, 3, "f32", backward=False)


def test_convnext_stage1_fwdbwd_full():
    """The benchmarked fwd+bwd workload: B=64 C=96 56x56, k=5, L=3, fp32."""
    check_full_size(64, 96, 56, 56, 5, 3, "f32", backward=True)


@pytest.mark.parametrize("L", [1, 2, 3, 4, 5])
def test_convnext_stage2_fwdbwd_full(L):
    """B=64 C=192 28x28, k=5, L sweep, fp32."""
    check_full_size(64, 192, 28, 28, 5, L, "f32", backward=True)


def test_convnext_stage1_bf16_l5_full():
    """B=128 C=96 56x56, k=5, L=5, bf16 storage."""
    check_full_size(128, 96, 56, 56, 5, 5, "bf16", backward=True)


# The shape sweep at every L = 1..5 in fp32 and bf16 (the 224 x 224 entry is
# test_large_224_fwdbwd_full): the planner's choices depend on B * C, so these
# full-size plans are not reached by the small shapes above.
SWEEP = [(128, 96, 56, 56), (128, 192, 28, 28), (128, 384, 14, 14), (128, 768, 7, 7), (32, 128, 63, 95)]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("L", [1, 2, 3, 4, 5])
@pytest.mark.parametrize("shape", SWEEP)
def test_sweep_fwdbwd(shape, L, dtype):
    B, C, H, W = shape
    check_full_size(B, C, H, W, 5, L, dtype, backward=True, n_planes=6, n_channels=2)


# One shape per execution path: the gradient pass (one block per thread), its
# block rounds, its coarse split, at L = 1, and the fused backward.
DETERMINISM = [
    (8, 12, 56, 56, 5, 3),
    (3, 16, 63, 95, 5, 3),
    (6, 20, 28, 28, 5, 5),
    (4, 6, 34, 30, 3, 1),
    (16, 20, 14, 14, 5, 2),
]


@pytest.mark.parametrize("B,C,H,W,k,L", DETERMINISM)
def test_determinism_bitwise(B, C, H, W, k, L):
    inp, dev = setup(B, C, H, W, k, L, "f32", seed=3)
    y1, y2 = dev.forward(), dev.forward()
    assert torch.equal(y1, y2)
    g1, g2 = dev.backward(), dev.backward()
    for a, b in zip([g1[0], g1[1], g1[2]] + g1[3] + g1[4], [g2[0], g2[1], g2[2]] + g2[3] + g2[4]):
        assert torch.equal(a, b)


def test_identity_pattern_reproduces_input():
    """Base zeroed, identity on LH/HL/HH at every level and on LL at level L only,
    unit scales: the operator returns x (up to fp32 rounding)."""
    B, C, H, W, k, L = 2, 3, 37, 29, 5, 4
    inp, dev = setup(B, C, H, W, k, L, "f32")
    dev.bw.zero_()
    for l in range(L):
        w = torch.zeros(4 * C, k, k, device="cuda:0")
        for c in range(C):
            for q in range(4):
                if q > 0 or l == L - 1:
                    w[4 * c + q, k // 2, k // 2] = 1.0
        dev.lw[l].copy_(w)
        dev.ls[l].fill_(1.0)
    y = to_np(dev.forward())
    assert rel_err(y, inp.x) < 1e-6


@pytest.mark.parametrize("B,C,H,W,k,L,dtype,with_bias", [(2, 3, 13, 11, 5, 3, "f32", False),
                                                          (1, 2, 130, 126, 5, 3, "f32", True),
                                                          (70, 3, 7, 6, 5, 4, "bf16", False)])
def test_prepared_forward_matches(B, C, H, W, k, L, dtype, with_bias):
    """binding.Forward (parameters validated once, workspace kept) gives
    bit-for-bit the output of binding.forward, on repeated calls and across
    inputs; it refuses activations of another shape before any library call."""
    from paper_2608_10805_amd import binding
    from paper_2608_10805_amd.inputs import make_bias

    inp, dev = setup(B, C, H, W, k, L, dtype)
    bias = torch.from_numpy(make_bias(C)).to("cuda:0") if with_bias else None
    fw = binding.Forward(dev.x, dev.bw, dev.bs, dev.lw, dev.ls, bias=bias)
    ref = binding.forward(dev.x, dev.bw, dev.bs, dev.lw, dev.ls, bias=bias)
    x2 = dev.x.flip(-1).contiguous()
    ref2 = binding.forward(x2, dev.bw, dev.bs, dev.lw, dev.ls, bias=bias)
    y = torch.empty_like(dev.x)
    for _ in range(2):
        assert torch.equal(fw.run(dev.x, y), ref)
        assert torch.equal(fw.run(x2, y), ref2)
    torch.cuda.synchronize()
    with pytest.raises(ValueError):
        fw.run(dev.x, torch.empty(B, C, H + 1, W, dtype=dev.x.dtype, device="cuda:0"))


def test_autograd_module_matches_binding():
    from paper_2608_10805_amd.autograd import WTConv2d

    torch.manual_seed(0)
    m = WTConv2d(6, kernel_size=5, levels=3, device="cuda:0")
    x = torch.randn(3, 6, 30, 26, device="cuda:0", requires_grad=True)
    y = m(x)
    g = torch.randn_like(y)
    y.backward(g)
    inp_x = x.detach().cpu().double().numpy()
    bw = m.base_w.detach().cpu().double().numpy()
    bs = m.base_scale.detach().cpu().double().numpy()
    lw = [p.detach().cpu().double().numpy() for p in m.level_w]
    ls = [p.detach().cpu().double().numpy() for p in m.level_scale]
    assert rel_err(to_np(y), oracle.forward(inp_x, bw, bs, lw, ls)) < 1e-5
    ref = oracle.backward(inp_x, g.cpu().double().numpy(), bw, bs, lw, ls)
    assert rel_err(to_np(x.grad), ref["dx"]) < 1e-5
    assert rel_err(to_np(m.base_w.grad), ref["d_base_w"]) < 1e-5
    for l in range(3):
        assert rel_err(to_np(m.level_w[l].grad), ref["d_level_w"][l]) < 1e-5
        assert rel_err(to_np(m.level_scale[l].grad), ref["d_level_scale"][l]) < 1e-5


# Planes of at most 8 x 8 pixels run in the tiny-plane kernels (one lane per
# batch entry, groups of 64): ragged batch groups, channel counts that are not
# multiples of four, every kernel size, L up to 8 and 16-bit storage.
TINY = [
    (70, 3, 7, 6, 5, 4, "f32"),
    (2, 5, 8, 8, 7, 8, "f32"),
    (65, 2, 5, 3, 1, 2, "f32"),
    (3, 4, 4, 7, 3, 3, "bf16"),
    (128, 9, 7, 7, 5, 5, "f16"),
    (1, 1, 2, 2, 5, 1, "f32"),
    (64, 4, 7, 7, 5, 0, "f32"),
]


@pytest.mark.parametrize("B,C,H,W,k,L,dtype", TINY)
def test_tiny_plane_forward(B, C, H, W, k, L, dtype):
    check_forward(B, C, H, W, k, L, dtype)


@pytest.mark.parametrize("B,C,H,W,k,L,dtype", TINY)
def test_tiny_plane_backward(B, C, H, W, k, L, dtype):
    check_backward(B, C, H, W, k, L, dtype)


def test_tiny_plane_backward_without_dx():
    check_backward(70, 3, 7, 6, 5, 4, "f32", need_dx=False)


# Resident planes with levels beyond the first 8 x 8 grid (level m) may run
# the coarse levels as a tiny sub-problem on the level-m carrier and the fused
# pass on levels 1..m with the coarse contribution added at level m (the
# backward pass splits more often than the forward): m = 1, 2, 3 and 4 in both
# passes, every kernel size, B above 64, 16-bit storage.
SPLIT = [
    (2, 3, 14, 14, 5, 3, "f32"),
    (2, 3, 14, 14, 5, 4, "f32"),
    (3, 2, 28, 28, 5, 4, "f32"),
    (2, 2, 20, 12, 3, 4, "f32"),
    (2, 2, 56, 56, 5, 5, "f32"),
    (1, 2, 63, 95, 5, 5, "f32"),
    (2, 3, 28, 28, 7, 3, "bf16"),
    (66, 2, 14, 14, 1, 2, "f16"),
    (2, 2, 28, 28, 5, 5, "f32"),
    (1, 2, 56, 56, 5, 6, "f32"),
    (1, 1, 63, 95, 3, 7, "f32"),
]


@pytest.mark.parametrize("B,C,H,W,k,L,dtype", SPLIT)
def test_split_forward(B, C, H, W, k, L, dtype):
    check_forward(B, C, H, W, k, L, dtype)


@pytest.mark.parametrize("B,C,H,W,k,L,dtype", SPLIT)
def test_split_backward(B, C, H, W, k, L, dtype):
    check_backward(B, C, H, W, k, L, dtype)


def test_split_backward_without_dx():
    check_backward(3, 2, 28, 28, 5, 4, "f32", need_dx=False)


@pytest.mark.parametrize("B,C,H,k,L,dtype", [(64, 192, 16, 5, 3, "f32"), (128, 192, 12, 5, 3, "bf16"),
                                             (128, 384, 14, 5, 3, "f16")])
def test_split_rule_shapes_full(B, C, H, k, L, dtype):
    """Forwards at the sizes where the split rule's plane-count threshold
    decides (too few planes to fill the chip: whole; B128 C384: split)."""
    check_full_size(B, C, H, H, k, L, dtype, backward=True, n_planes=6, n_channels=2)


@pytest.mark.parametrize("B,C,H,L,dtype", [(96, 192, 18, 3, "bf16"), (128, 192, 26, 3, "f32"),
                                           (64, 192, 20, 3, "f32")])
def test_grad_shed_one_level_full(B, C, H, L, dtype):
    """Backwards around the plane count from which the gradient pass sheds a
    single level above m = 2 to the coarse sub-problem (B96 and B128 C192:
    shed; B64 C192: whole)."""
    check_full_size(B, C, H, H, 5, L, dtype, backward=True, n_planes=6, n_channels=2)


# Planes whose working set does not fit one compute unit's LDS take the split
# path: the coarse levels run on the level-1 carrier (recursively, if that is
# still too large) and the base path plus level 1 run on halo tiles. Every
# element is checked; the cases cover a split in the backward pass only, in
# both passes, k = 1 (no halo), k = 7, L = 0 and 1 (no carrier), a two-deep
# recursion, ragged tiles and 16-bit storage.
LARGE = [
    (2, 2, 100, 100, 5, 3, "f32"),
    (1, 2, 130, 126, 5, 3, "f32"),
    (1, 3, 130, 70, 1, 2, "f32"),
    (2, 3, 90, 90, 7, 1, "f32"),
    (1, 2, 150, 130, 3, 0, "f32"),
    (1, 2, 224, 224, 5, 5, "f32"),
    (1, 1, 300, 300, 7, 4, "f32"),
    (1, 2, 190, 170, 5, 4, "f32"),
    (1, 2, 224, 224, 5, 3, "bf16"),
    (1, 2, 190, 170, 5, 4, "f16"),
]


@pytest.mark.parametrize("B,C,H,W,k,L,dtype", LARGE)
def test_large_plane_forward(B, C, H, W, k, L, dtype):
    check_forward(B, C, H, W, k, L, dtype)


@pytest.mark.parametrize("B,C,H,W,k,L,dtype", LARGE)
def test_large_plane_backward(B, C, H, W, k, L, dtype):
    check_backward(B, C, H, W, k, L, dtype)


def test_large_plane_backward_without_dx():
    check_backward(2, 2, 100, 100, 5, 3, "f32", need_dx=False)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("L", [1, 2, 3, 4, 5])
def test_large_224_fwdbwd_full(L, dtype):
    """B=16 C=64 224x224, k=5, L sweep (the large entry of the shape sweep)."""
    check_full_size(16, 64, 224, 224, 5, L, dtype, backward=True, n_planes=6, n_channels=2)


@pytest.mark.parametrize("C,H,L,dtype", [(32, 512, 5, "f32"), (32, 256, 3, "f16"), (64, 128, 1, "f32"),
                                         (32, 512, 2, "f16")])
def test_paper_layer_sweep_full(C, H, L, dtype):
    """The paper's layer sweep shapes (B=8, C in {32, 64, 128}, H=W in {128, 256, 512})."""
    check_full_size(8, C, H, H, 5, L, dtype, backward=True, n_planes=4, n_channels=2)


@pytest.mark.parametrize("C,H,k,L,dtype", [(64, 256, 3, 3, "f32"), (32, 512, 3, 5, "f16"), (64, 256, 7, 3, "f32"),
                                           (128, 128, 7, 4, "bf16"), (32, 512, 7, 2, "f32"),
                                           (128, 128, 3, 1, "f16")])
def test_paper_layer_sweep_other_k_full(C, H, k, L, dtype):
    """The paper's sweep shapes at k = 3 (its k = 3 table) and k = 7 (its
    traffic-invariance configurations), B = 8, forward and backward."""
    check_full_size(8, C, H, H, k, L, dtype, backward=True, n_planes=4, n_channels=2)


def test_large_plane_determinism_bitwise():
    inp, dev = setup(2, 3, 150, 150, 5, 3, "f32", seed=5)
    y1, y2 = dev.forward(), dev.forward()
    assert torch.equal(y1, y2)
    g1, g2 = dev.backward(), dev.backward()
    for a, b in zip([g1[0], g1[1], g1[2]] + g1[3] + g1[4], [g2[0], g2[1], g2[2]] + g2[3] + g2[4]):
        assert torch.equal(a, b)


# k = 9 (the largest kernel the boundary takes; the paper's experiments stop
# at 7), one shape per execution path: tiny planes, 8 x 8 planes whose tiny
# backward LDS would not fit (resident with mixed rounds instead), mixed
# forward rounds, forward regions on small planes, the split backward, the
# gradient pass with one block per thread and with block rounds, the region
# gradient route, L = 0 and a deep split. At k = 9 a kernel row has 81 taps,
# more than a wavefront's lanes: the finalize wraps them round the lanes and
# the tiny backward flushes its gradient queue within one kernel.
K9 = [
    (70, 3, 7, 6, 9, 4, "f32"),
    (2, 3, 7, 7, 9, 3, "bf16"),
    (2, 3, 8, 8, 9, 8, "f32"),
    (2, 3, 14, 14, 9, 2, "f32"),
    (16, 8, 16, 16, 9, 3, "f32"),
    (2, 3, 28, 28, 9, 3, "f16"),
    (2, 3, 40, 40, 9, 3, "f32"),
    (2, 2, 56, 56, 9, 3, "f32"),
    (2, 2, 63, 95, 9, 4, "f32"),
    (1, 2, 130, 126, 9, 3, "f32"),
    (1, 2, 150, 140, 9, 1, "bf16"),
    (2, 3, 14, 14, 9, 0, "f32"),
    (2, 3, 28, 28, 9, 1, "bf16"),
    (66, 2, 14, 14, 9, 5, "f32"),
]


@pytest.mark.parametrize("B,C,H,W,k,L,dtype", K9)
def test_k9_forward(B, C, H, W, k, L, dtype):
    check_forward(B, C, H, W, k, L, dtype)


@pytest.mark.parametrize("B,C,H,W,k,L,dtype", K9)
def test_k9_backward(B, C, H, W, k, L, dtype):
    check_backward(B, C, H, W, k, L, dtype)


@pytest.mark.parametrize("B,C,H,W,k,L,dtype", [(2, 4, 28, 28, 9, 3, "f32"), (70, 3, 7, 6, 9, 4, "f32"),
                                                (1, 2, 130, 126, 9, 3, "f32")])
def test_k9_bias(B, C, H, W, k, L, dtype):
    test_bias_forward_backward(B, C, H, W, k, L, dtype)


# Large planes at k = 7: the region gradient route over 48 x 48 tiles
# (ragged tiles, a coarse sub-problem or none, 16-bit storage); at L = 0 the
# fused region backward runs.
K7_REGION = [
    (1, 2, 130, 126, 7, 3, "f32"),
    (2, 3, 150, 140, 7, 2, "bf16"),
    (1, 3, 129, 131, 7, 1, "f16"),
    (1, 2, 130, 126, 7, 4, "f32"),
    (1, 2, 130, 126, 5, 0, "f32"),
    (1, 2, 130, 126, 7, 0, "bf16"),
]


@pytest.mark.parametrize("B,C,H,W,k,L,dtype", K7_REGION)
def test_k7_region_backward(B, C, H, W, k, L, dtype):
    check_backward(B, C, H, W, k, L, dtype)


def test_k7_region_full_size():
    check_full_size(16, 64, 224, 224, 7, 3, "f32", backward=True)


def test_k9_determinism_bitwise():
    test_determinism_bitwise(4, 6, 56, 56, 9, 3)


@pytest.mark.parametrize("B,C,H,W,L,dtype", [(32, 64, 56, 56, 3, "f32"), (128, 384, 14, 14, 4, "bf16")])
def test_k9_full_size(B, C, H, W, L, dtype):
    check_full_size(B, C, H, W, 9, L, dtype, backward=True)


def _random_cases(seed, n):
    """Seeded random shapes across every execution path: tiny, resident with one
    or several planes, split, gradient pass (one block per thread or block
    rounds), fused backward; odd, even and 4-multiple widths; all k, L and
    storage types."""
    import random
    rng = random.Random(seed)
    sizes = [1, 2, 3, 5, 7, 8, 9, 12, 14, 15, 16, 17, 20, 23, 28, 30, 31, 33, 40, 46, 47, 56, 63, 64, 66, 70, 95, 97]
    cases = []
    for _ in range(n):
        cases.append((rng.choice([1, 2, 3, 5, 7, 9, 16]), rng.choice([1, 2, 3, 4, 8, 64, 130]), rng.choice(sizes),
                      rng.choice(sizes), rng.choice([1, 3, 5, 7]), rng.choice([0, 1, 2, 3, 4, 5, 6]),
                      rng.choice(["f32", "f32", "bf16", "f16"])))
    return cases


@pytest.mark.parametrize("B,C,H,W,k,L,dtype", _random_cases(2026, 180))
def test_random_shapes(B, C, H, W, k, L, dtype):
    check_forward(B, C, H, W, k, L, dtype)
    check_backward(B, C, H, W, k, L, dtype)
