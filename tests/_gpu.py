"""Helpers for the GPU parity tests: run the library through the C ABI on
seeded inputs and compare with the float64 oracle on the same values."""
import numpy as np
import torch

from paper_2608_10805_amd import binding
from paper_2608_10805_amd.inputs import make_inputs

TORCH_DTYPE = {"f32": torch.float32, "bf16": torch.bfloat16, "f16": torch.float16}
TOL = {"f32": 1e-5, "bf16": 2e-2, "f16": 2e-2}


def rel_err(got, want):
    """max |got - want| / max |want| over the tensor (float64)."""
    got = np.asarray(got, dtype=np.float64)
    want = np.asarray(want, dtype=np.float64)
    assert got.shape == want.shape, (got.shape, want.shape)
    return float(np.abs(got - want).max() / max(np.abs(want).max(), 1e-30))


class Dev:
    """Inputs resident on the GPU (activations in the storage dtype, parameters fp32)."""

    def __init__(self, inp, dtype, device="cuda:0"):
        self.inp = inp
        self.dtype = dtype
        td = TORCH_DTYPE[dtype]
        f32 = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(device)  # noqa: E731
        self.x = f32(inp.x).to(td).contiguous()
        self.dy = f32(inp.dy).to(td).contiguous() if inp.dy is not None else None
        self.bw, self.bs = f32(inp.base_w), f32(inp.base_scale)
        self.lw = [f32(a) for a in inp.level_w]
        self.ls = [f32(a) for a in inp.level_scale]

    def forward(self):
        y = binding.forward(self.x, self.bw, self.bs, self.lw, self.ls)
        torch.cuda.synchronize()
        return y

    def backward(self, need_dx=True):
        out = binding.backward(self.x, self.dy, self.bw, self.bs, self.lw, self.ls, need_dx=need_dx)
        torch.cuda.synchronize()
        return out


def to_np(t):
    return t.detach().float().cpu().numpy().astype(np.float64)


def setup(B, C, H, W, k, L, dtype, seed=0):
    inp = make_inputs(B, C, H, W, k, L, dtype, seed=seed, with_dy=True)
    return inp, Dev(inp, dtype)


def channel_slice(inp, cs):
    """Inputs restricted to channels cs (all batch entries), for oracle checks of
    parameter gradients, which only couple planes of the same channel."""
    cs = np.asarray(cs)
    lw = [w.reshape(-1, 4, *w.shape[1:])[cs].reshape(-1, *w.shape[1:]) for w in inp.level_w]
    ls = [s.reshape(-1, 4)[cs].reshape(-1) for s in inp.level_scale]
    return (inp.x[:, cs], inp.dy[:, cs], inp.base_w[cs], inp.base_scale[cs], lw, ls)
