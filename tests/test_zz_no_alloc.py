"""wtconv_backward_noalloc (the backward with the library's static scratch as
its workspace) against wtconv_backward with a caller's workspace, through the
C ABI: two calls in a row on one GPU, the second on a smaller problem, so the
second runs over whatever the first left in the shared scratch. The kernels
are the same, so the results must agree bit for bit."""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

from paper_2608_10805_amd import binding  # noqa: E402
from paper_2608_10805_amd.inputs import make_bias, make_inputs  # noqa: E402

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():
    pytest.skip("needs a GPU", allow_module_level=True)

DEV = "cuda:0"
TD = {"f32": torch.float32, "bf16": torch.bfloat16, "f16": torch.float16}


def _problem(B, C, H, W, k, L, dtype, seed):
    inp = make_inputs(B, C, H, W, k, L, dtype, seed=seed)
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(DEV)  # noqa: E731
    p = {"x": t(inp.x).to(TD[dtype]), "dy": t(inp.dy).to(TD[dtype]), "bw": t(inp.base_w), "bs": t(inp.base_scale),
         "b0": t(make_bias(C, seed)), "lw": [t(a) for a in inp.level_w], "ls": [t(a) for a in inp.level_scale]}
    p["desc"] = binding.make_desc(B, C, H, W, k, L, binding._dtype_code(p["x"]))
    return p


def _outputs(p):
    o = {"dx": torch.full_like(p["x"], float("nan")), "dbw": torch.full_like(p["bw"], float("nan")),
         "dbs": torch.full_like(p["bs"], float("nan")), "dbb": torch.full_like(p["bs"], float("nan")),
         "dlw": [torch.full_like(a, float("nan")) for a in p["lw"]],
         "dls": [torch.full_like(a, float("nan")) for a in p["ls"]]}
    return o


def _args(p, o):
    ptr = lambda ts: [a.data_ptr() for a in ts]  # noqa: E731
    return (p["desc"], p["x"].data_ptr(), p["dy"].data_ptr(), p["bw"].data_ptr(), p["bs"].data_ptr(),
            p["b0"].data_ptr(), ptr(p["lw"]), ptr(p["ls"]), o["dx"].data_ptr(), o["dbw"].data_ptr(),
            o["dbs"].data_ptr(), o["dbb"].data_ptr(), ptr(o["dlw"]), ptr(o["dls"]))


def _with_workspace(p):
    o = _outputs(p)
    n = binding.wtconv_backward_workspace_bytes(p["desc"])
    ws = torch.empty(n, dtype=torch.uint8, device=DEV)
    rc = binding.wtconv_backward(*_args(p, o), ws.data_ptr(), n, torch.cuda.current_stream().cuda_stream)
    assert rc == 0, binding.status_string(rc)
    return o


def _noalloc(p):
    o = _outputs(p)
    rc = binding.wtconv_backward_noalloc(*_args(p, o), torch.cuda.current_stream().cuda_stream)
    assert rc == 0, binding.status_string(rc)
    return o


def _flat(o):
    return [o["dx"], o["dbw"], o["dbs"], o["dbb"]] + o["dlw"] + o["dls"]


# (first problem, second smaller problem): the gradient pass with dx from the
# rotated forward, then a fused backward; a split whose carriers live in the
# scratch, then tiny planes.
PAIRS = [
    ((64, 96, 56, 56, 5, 3, "f32"), (4, 8, 28, 28, 5, 4, "bf16")),
    ((32, 384, 14, 14, 5, 3, "f32"), (70, 6, 7, 7, 3, 2, "f16")),
]


@pytest.mark.parametrize("first,second", PAIRS)
def test_noalloc_matches_backward_on_two_calls(first, second):
    for seed, shape in enumerate((first, second)):
        print(f"noalloc: B,C,H,W,k,L,dtype = {shape}", flush=True)
        p = _problem(*shape, seed=seed)
        assert 0 < binding.wtconv_backward_workspace_bytes(p["desc"]) <= binding.NOALLOC_SCRATCH_BYTES
        ref = _with_workspace(p)
        got = _noalloc(p)
        torch.cuda.synchronize()
        for a, b in zip(_flat(got), _flat(ref)):
            assert not torch.isnan(a).any()
            assert torch.equal(a, b)
