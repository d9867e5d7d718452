"""Host-side argument checks of the Python binding (no GPU, no library call):
every tensor an entry point receives is checked against the problem that x
defines before anything reaches the C ABI, which sees only pointers and the
descriptor. Each rejection is exercised with CPU tensors (validate(...,
on_gpu=False)); the entry points themselves refuse CPU tensors outright."""
import pytest

torch = pytest.importorskip("torch")

from paper_2608_10805_amd import binding  # noqa: E402


def problem(B=2, C=3, H=9, W=7, k=5, L=2, dtype=torch.float32):
    f = torch.float32
    x = torch.zeros(B, C, H, W, dtype=dtype)
    return dict(x=x, base_w=torch.zeros(C, k, k, dtype=f), base_scale=torch.zeros(C, dtype=f),
                level_w=[torch.zeros(4 * C, k, k, dtype=f) for _ in range(L)],
                level_scale=[torch.zeros(4 * C, dtype=f) for _ in range(L)])


def check(**kw):
    return binding.validate(on_gpu=False, **kw)


def test_a_consistent_problem_passes():
    p = problem()
    assert check(**p, bias=torch.zeros(3), out=torch.zeros(2, 3, 9, 7), dy=torch.zeros(2, 3, 9, 7)) == \
        (2, 3, 9, 7, 5, 2)
    assert check(**problem(L=0)) == (2, 3, 9, 7, 5, 0)
    assert check(**problem(dtype=torch.bfloat16)) == (2, 3, 9, 7, 5, 2)


@pytest.mark.parametrize("mutate,match", [
    (lambda p: p.update(x=torch.zeros(3, 9, 7)), r"\[B, C, H, W\]"),
    (lambda p: p.update(x=torch.zeros(2, 3, 0, 7)), "empty"),
    (lambda p: p.update(x=torch.zeros(2, 3, 9, 7, dtype=torch.float64)), "float32, bfloat16 or float16"),
    (lambda p: p.update(x=torch.zeros(2, 3, 7, 9).transpose(2, 3)), "contiguous"),
    (lambda p: p.update(base_w=torch.zeros(3, 4, 4)), "odd"),
    (lambda p: p.update(base_w=torch.zeros(3, 5, 3)), r"\[C, k, k\]"),
    (lambda p: p.update(base_w=torch.zeros(4, 5, 5)), "base_w must have shape"),
    (lambda p: p.update(base_w=torch.zeros(3, 5, 5, dtype=torch.float64)), "base_w must be torch.float32"),
    (lambda p: p.update(base_scale=torch.zeros(2)), "base_scale must have shape"),
    (lambda p: p.update(base_scale=torch.zeros(3, dtype=torch.float16)), "base_scale must be torch.float32"),
    (lambda p: p["level_w"].pop(), "level_w has 1 levels but level_scale has 2"),
    (lambda p: p["level_scale"].pop(), "level_w has 2 levels but level_scale has 1"),
    (lambda p: p["level_w"].__setitem__(1, torch.zeros(3, 5, 5)), r"level_w\[1\] must have shape"),
    (lambda p: p["level_w"].__setitem__(0, torch.zeros(12, 3, 3)), r"level_w\[0\] must have shape"),
    (lambda p: p["level_scale"].__setitem__(0, torch.zeros(3)), r"level_scale\[0\] must have shape"),
    (lambda p: p.update(level_w=[torch.zeros(12, 5, 5)] * 9, level_scale=[torch.zeros(12)] * 9), "at most 8"),
])
def test_rejections(mutate, match):
    p = problem()
    mutate(p)
    with pytest.raises(ValueError, match=match):
        check(**p)


@pytest.mark.parametrize("name,bad,match", [
    ("bias", torch.zeros(4), "bias must have shape"),
    ("out", torch.zeros(2, 3, 9, 8), "out must have shape"),
    ("out", torch.zeros(2, 3, 9, 7, dtype=torch.bfloat16), "out must be torch.float32"),
    ("dy", torch.zeros(1, 3, 9, 7), "dy must have shape"),
    ("dy", torch.zeros(2, 3, 9, 7, dtype=torch.float16), "dy must be torch.float32"),
])
def test_optional_tensor_rejections(name, bad, match):
    with pytest.raises(ValueError, match=match):
        check(**problem(), **{name: bad})


def test_entry_points_refuse_host_tensors_before_any_library_call():
    p = problem()
    with pytest.raises(ValueError, match="GPU tensor"):
        binding.forward(p["x"], p["base_w"], p["base_scale"], p["level_w"], p["level_scale"])
    with pytest.raises(ValueError, match="GPU tensor"):
        binding.backward(p["x"], p["x"], p["base_w"], p["base_scale"], p["level_w"], p["level_scale"])
    with pytest.raises(ValueError, match="GPU tensor"):
        binding.backward_data(p["x"], p["base_w"], p["base_scale"], p["level_w"], p["level_scale"])


@pytest.mark.parametrize("call", ["forward", "backward", "partials", "finalize", "data"])
def test_raw_calls_need_one_pointer_per_level(call):
    """The C side reads desc.L pointers from each host array, so a list of
    another length is refused before the call (nothing is dereferenced)."""
    desc = binding.make_desc(1, 1, 8, 8, 5, 2)
    short, full = [1 << 40], [1 << 40, (1 << 40) + 64]
    with pytest.raises(ValueError, match="L = 2"):
        if call == "forward":
            binding.wtconv_forward(desc, 1, 1, 1, None, full, short, 1, None, 0, None)
        elif call == "backward":
            binding.wtconv_backward(desc, 1, 1, 1, 1, None, full, full, 1, 1, 1, None, full, short, 1, 1, None)
        elif call == "partials":
            binding.wtconv_backward_partials(desc, 1, 1, 1, 1, short, full, 1, 1, 1, None)
        elif call == "finalize":
            binding.wtconv_backward_finalize(desc, 1, 1, None, full, full, 1, 1, None, short, full, 1, 1, None)
        else:
            binding.wtconv_backward_data(desc, 1, 1, 1, full, None, 1, 1, 1, None)
