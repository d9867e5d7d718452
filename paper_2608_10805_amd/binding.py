"""ctypes binding of libwtconv.so (include/wtconv.h), with the same entry-point names.

This module only marshals arguments: every step of the operator runs in the
library's HIP kernels. torch is used for device memory and the current HIP
stream. If the library is missing, loading fails loudly; there is no CPU
fallback.
"""
import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libwtconv.so")

WTCONV_F32, WTCONV_BF16, WTCONV_F16 = 0, 1, 2
STATUS = {
    0: "WTCONV_OK", 1: "WTCONV_ERR_NULL", 2: "WTCONV_ERR_SHAPE", 3: "WTCONV_ERR_KSIZE",
    4: "WTCONV_ERR_LEVELS", 5: "WTCONV_ERR_DTYPE", 6: "WTCONV_ERR_ALIAS", 7: "WTCONV_ERR_WORKSPACE",
    8: "WTCONV_ERR_UNSUPPORTED", 9: "WTCONV_ERR_HIP", 10: "WTCONV_ERR_SCRATCH",
}
EXPORTS = ["wtconv_forward_workspace_bytes", "wtconv_forward", "wtconv_backward", "wtconv_backward_workspace_bytes",
           "wtconv_backward_partials", "wtconv_backward_finalize", "wtconv_backward_data_workspace_bytes",
           "wtconv_backward_data", "wtconv_backward_noalloc", "wtconv_status_string", "wtconv_version"]
NOALLOC_SCRATCH_BYTES = 64 << 20  # WTCONV_NOALLOC_SCRATCH_BYTES
MAX_LEVELS = 8


class WTConvError(RuntimeError):
    def __init__(self, status, msg):
        super().__init__(f"{STATUS.get(status, status)}: {msg}")
        self.status = status


class Desc(ctypes.Structure):
    _fields_ = [("B", ctypes.c_int), ("C", ctypes.c_int), ("H", ctypes.c_int), ("W", ctypes.c_int),
                ("k", ctypes.c_int), ("L", ctypes.c_int), ("dtype", ctypes.c_int)]


_lib = None
_P = ctypes.c_void_p
_PP = ctypes.POINTER(ctypes.c_void_p)


def load():
    """Load the in-tree library (building it first only if it was never built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        from . import build
        build.build()
    lib = ctypes.CDLL(LIB_PATH)
    lib.wtconv_forward_workspace_bytes.argtypes = [ctypes.POINTER(Desc)]
    lib.wtconv_forward_workspace_bytes.restype = ctypes.c_size_t
    lib.wtconv_forward.argtypes = [ctypes.POINTER(Desc), _P, _P, _P, _P, _PP, _PP, _P, _P, ctypes.c_size_t, _P]
    lib.wtconv_forward.restype = ctypes.c_int
    lib.wtconv_backward_workspace_bytes.argtypes = [ctypes.POINTER(Desc)]
    lib.wtconv_backward_workspace_bytes.restype = ctypes.c_size_t
    lib.wtconv_backward.argtypes = [ctypes.POINTER(Desc), _P, _P, _P, _P, _P, _PP, _PP, _P, _P, _P, _P, _PP, _PP,
                                    _P, ctypes.c_size_t, _P]
    lib.wtconv_backward.restype = ctypes.c_int
    lib.wtconv_backward_partials.argtypes = [ctypes.POINTER(Desc), _P, _P, _P, _P, _PP, _PP, _P, _P,
                                             ctypes.c_size_t, _P]
    lib.wtconv_backward_partials.restype = ctypes.c_int
    lib.wtconv_backward_finalize.argtypes = [ctypes.POINTER(Desc), _P, _P, _P, _PP, _PP, _P, _P, _P, _PP, _PP,
                                             _P, ctypes.c_size_t, _P]
    lib.wtconv_backward_finalize.restype = ctypes.c_int
    lib.wtconv_backward_data_workspace_bytes.argtypes = [ctypes.POINTER(Desc)]
    lib.wtconv_backward_data_workspace_bytes.restype = ctypes.c_size_t
    lib.wtconv_backward_data.argtypes = [ctypes.POINTER(Desc), _P, _P, _P, _PP, _PP, _P, _P, ctypes.c_size_t, _P]
    lib.wtconv_backward_data.restype = ctypes.c_int
    lib.wtconv_backward_noalloc.argtypes = [ctypes.POINTER(Desc), _P, _P, _P, _P, _P, _PP, _PP, _P, _P, _P, _P,
                                            _PP, _PP, _P]
    lib.wtconv_backward_noalloc.restype = ctypes.c_int
    lib.wtconv_status_string.argtypes = [ctypes.c_int]
    lib.wtconv_status_string.restype = ctypes.c_char_p
    lib.wtconv_version.restype = ctypes.c_int
    _lib = lib
    return lib


def status_string(status: int) -> str:
    return load().wtconv_status_string(status).decode()


def _check(rc):
    if rc != 0:
        raise WTConvError(rc, status_string(rc))


def make_desc(B, C, H, W, k, L, dtype=WTCONV_F32) -> Desc:
    return Desc(int(B), int(C), int(H), int(W), int(k), int(L), int(dtype))


def _level_lists(desc, **lists):
    """The C entry points read desc.L pointers from each host array: every
    list must hold exactly that many (an L = 0 problem may pass None)."""
    for name, v in lists.items():
        n = 0 if v is None else len(v)
        if n != desc.L:
            raise ValueError(f"{name} has {n} entries but the descriptor has L = {desc.L}")


def _ptr_array(ptrs):
    n = max(len(ptrs), 1)
    arr = (ctypes.c_void_p * n)(*([ctypes.c_void_p(p) for p in ptrs] or [None]))
    return arr if ptrs else None


# ----------------------------------------------------------------------------
# raw entry points (integers as device addresses)
# ----------------------------------------------------------------------------

def wtconv_forward_workspace_bytes(desc: Desc) -> int:
    return int(load().wtconv_forward_workspace_bytes(ctypes.byref(desc)))


def wtconv_forward(desc: Desc, x, base_w, base_scale, base_bias, level_w, level_scale, y, workspace,
                   workspace_bytes, stream) -> int:
    """Raw call: pointers are integers (device addresses, base_bias may be None);
    level_* are lists of desc.L addresses."""
    _level_lists(desc, level_w=level_w, level_scale=level_scale)
    return load().wtconv_forward(ctypes.byref(desc), x, base_w, base_scale, base_bias, _ptr_array(level_w),
                                 _ptr_array(level_scale), y, workspace, ctypes.c_size_t(workspace_bytes), stream)


def wtconv_backward_workspace_bytes(desc: Desc) -> int:
    return int(load().wtconv_backward_workspace_bytes(ctypes.byref(desc)))


def wtconv_backward(desc: Desc, x, dy, base_w, base_scale, base_bias, level_w, level_scale, dx, d_base_w,
                    d_base_scale, d_base_bias, d_level_w, d_level_scale, workspace, workspace_bytes, stream) -> int:
    _level_lists(desc, level_w=level_w, level_scale=level_scale, d_level_w=d_level_w, d_level_scale=d_level_scale)
    return load().wtconv_backward(ctypes.byref(desc), x, dy, base_w, base_scale, base_bias, _ptr_array(level_w),
                                  _ptr_array(level_scale), dx, d_base_w, d_base_scale, d_base_bias,
                                  _ptr_array(d_level_w), _ptr_array(d_level_scale), workspace,
                                  ctypes.c_size_t(workspace_bytes), stream)


def wtconv_backward_noalloc(desc: Desc, x, dy, base_w, base_scale, base_bias, level_w, level_scale, dx, d_base_w,
                            d_base_scale, d_base_bias, d_level_w, d_level_scale, stream) -> int:
    """wtconv_backward with the library's static scratch as its workspace."""
    _level_lists(desc, level_w=level_w, level_scale=level_scale, d_level_w=d_level_w, d_level_scale=d_level_scale)
    return load().wtconv_backward_noalloc(ctypes.byref(desc), x, dy, base_w, base_scale, base_bias,
                                          _ptr_array(level_w), _ptr_array(level_scale), dx, d_base_w, d_base_scale,
                                          d_base_bias, _ptr_array(d_level_w), _ptr_array(d_level_scale), stream)


def wtconv_backward_partials(desc: Desc, x, dy, base_w, base_scale, level_w, level_scale, dx, workspace,
                             workspace_bytes, stream) -> int:
    _level_lists(desc, level_w=level_w, level_scale=level_scale)
    return load().wtconv_backward_partials(ctypes.byref(desc), x, dy, base_w, base_scale, _ptr_array(level_w),
                                           _ptr_array(level_scale), dx, workspace,
                                           ctypes.c_size_t(workspace_bytes), stream)


def wtconv_backward_finalize(desc: Desc, base_w, base_scale, base_bias, level_w, level_scale, d_base_w,
                             d_base_scale, d_base_bias, d_level_w, d_level_scale, workspace, workspace_bytes,
                             stream) -> int:
    _level_lists(desc, level_w=level_w, level_scale=level_scale, d_level_w=d_level_w, d_level_scale=d_level_scale)
    return load().wtconv_backward_finalize(ctypes.byref(desc), base_w, base_scale, base_bias, _ptr_array(level_w),
                                           _ptr_array(level_scale), d_base_w, d_base_scale, d_base_bias,
                                           _ptr_array(d_level_w), _ptr_array(d_level_scale), workspace,
                                           ctypes.c_size_t(workspace_bytes), stream)


def wtconv_backward_data_workspace_bytes(desc: Desc) -> int:
    return int(load().wtconv_backward_data_workspace_bytes(ctypes.byref(desc)))


def wtconv_backward_data(desc: Desc, dy, base_w, base_scale, level_w, level_scale, dx, workspace, workspace_bytes,
                         stream) -> int:
    _level_lists(desc, level_w=level_w, level_scale=level_scale)
    return load().wtconv_backward_data(ctypes.byref(desc), dy, base_w, base_scale, _ptr_array(level_w),
                                       _ptr_array(level_scale), dx, workspace, ctypes.c_size_t(workspace_bytes),
                                       stream)


def wtconv_version() -> int:
    return int(load().wtconv_version())


# ----------------------------------------------------------------------------
# torch-tensor conveniences (marshalling only)
# ----------------------------------------------------------------------------

def _dtype_code(t):
    import torch
    return {torch.float32: WTCONV_F32, torch.bfloat16: WTCONV_BF16, torch.float16: WTCONV_F16}[t.dtype]


def _require(t, name, dtype=None, shape=None, device=None, on_gpu=True):
    import torch
    if not isinstance(t, torch.Tensor):
        raise ValueError(f"{name} must be a tensor")
    if on_gpu and not t.is_cuda:
        raise ValueError(f"{name} must be a GPU tensor")
    if device is not None and t.device != device:
        raise ValueError(f"{name} is on {t.device}, expected {device}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")


def validate(x, base_w, base_scale, level_w, level_scale, bias=None, out=None, dy=None, on_gpu=True):
    """Check every tensor the entry points receive against the problem x
    defines, before anything reaches the library (which sees only pointers
    and the descriptor): x [B,C,H,W] in fp32 / bf16 / fp16; base_w [C,k,k]
    with k odd; base_scale (and bias, if given) [C]; level_w and level_scale
    lists of the same length L <= 8 holding [4C,k,k] and [4C]; parameters
    fp32; out and dy (if given) of x's shape and dtype; everything contiguous
    and on x's device. Raises ValueError; returns (B, C, H, W, k, L)."""
    import torch
    _require(x, "x", on_gpu=on_gpu)
    if x.dtype not in (torch.float32, torch.bfloat16, torch.float16):
        raise ValueError(f"x must be float32, bfloat16 or float16, got {x.dtype}")
    if x.dim() != 4:
        raise ValueError(f"x must be [B, C, H, W], got shape {tuple(x.shape)}")
    B, C, H, W = x.shape
    if min(B, C, H, W) < 1:
        raise ValueError(f"x has an empty dimension: {tuple(x.shape)}")
    dev = x.device
    if not isinstance(base_w, torch.Tensor) or base_w.dim() != 3 or base_w.shape[1] != base_w.shape[2]:
        raise ValueError("base_w must be a [C, k, k] tensor")
    k = base_w.shape[-1]
    if k % 2 == 0:
        raise ValueError(f"the kernel size must be odd, got {k}")
    f32 = torch.float32
    _require(base_w, "base_w", f32, (C, k, k), dev, on_gpu)
    _require(base_scale, "base_scale", f32, (C,), dev, on_gpu)
    if bias is not None:
        _require(bias, "bias", f32, (C,), dev, on_gpu)
    level_w, level_scale = list(level_w), list(level_scale)
    if len(level_w) != len(level_scale):
        raise ValueError(f"level_w has {len(level_w)} levels but level_scale has {len(level_scale)}")
    if len(level_w) > MAX_LEVELS:
        raise ValueError(f"at most {MAX_LEVELS} levels, got {len(level_w)}")
    for i, (w, sc) in enumerate(zip(level_w, level_scale)):
        _require(w, f"level_w[{i}]", f32, (4 * C, k, k), dev, on_gpu)
        _require(sc, f"level_scale[{i}]", f32, (4 * C,), dev, on_gpu)
    if out is not None:
        _require(out, "out", x.dtype, x.shape, dev, on_gpu)
    if dy is not None:
        _require(dy, "dy", x.dtype, x.shape, dev, on_gpu)
    return B, C, H, W, k, len(level_w)


def _workspace_ok(ws, nbytes, device):
    """A caller-provided workspace is used only if it is a contiguous device
    tensor on the problem's device with at least nbytes bytes."""
    import torch
    return (isinstance(ws, torch.Tensor) and ws.device == device and ws.is_contiguous()
            and ws.numel() * ws.element_size() >= nbytes)


def _stream(device):
    import torch
    return torch.cuda.current_stream(device).cuda_stream


def forward(x, base_w, base_scale, level_w, level_scale, out=None, workspace=None, bias=None):
    """y = WTConv(x) on the current stream. x: [B,C,H,W] fp32/bf16/fp16 on the GPU;
    base_w [C,k,k], base_scale [C], level_w list of [4C,k,k], level_scale list of [4C] (fp32);
    bias: the base bias [C] (fp32) or None.
    Large planes need a device workspace; one is allocated if `workspace` is None or too small."""
    import torch
    B, C, H, W, k, L = validate(x, base_w, base_scale, level_w, level_scale, bias=bias, out=out)
    y = torch.empty_like(x) if out is None else out
    desc = make_desc(B, C, H, W, k, L, _dtype_code(x))
    nbytes = wtconv_forward_workspace_bytes(desc)
    ws_ptr = None
    if nbytes:
        if not _workspace_ok(workspace, nbytes, x.device):
            workspace = torch.empty(nbytes, dtype=torch.uint8, device=x.device)
        ws_ptr = workspace.data_ptr()
    _check(wtconv_forward(desc, x.data_ptr(), base_w.data_ptr(), base_scale.data_ptr(),
                          bias.data_ptr() if bias is not None else None,
                          [t.data_ptr() for t in level_w], [t.data_ptr() for t in level_scale], y.data_ptr(),
                          ws_ptr, nbytes, _stream(x.device)))
    return y


def backward(x, dy, base_w, base_scale, level_w, level_scale, need_dx=True, workspace=None, bias=None,
             need_dbias=False):
    """Gradients of sum(y * dy). Returns (dx or None, d_base_w, d_base_scale, [d_level_w], [d_level_scale]),
    followed by d_bias when need_dbias. `bias` (the base bias [C] or None) enters d_base_scale."""
    import torch
    B, C, H, W, k, L = validate(x, base_w, base_scale, level_w, level_scale, bias=bias, dy=dy)
    desc = make_desc(B, C, H, W, k, L, _dtype_code(x))
    nbytes = wtconv_backward_workspace_bytes(desc)
    if nbytes == 0:
        raise WTConvError(8, "no backward plan for this shape")
    if not _workspace_ok(workspace, nbytes, x.device):
        workspace = torch.empty(nbytes, dtype=torch.uint8, device=x.device)
    dx = torch.empty_like(x) if need_dx else None
    dbw = torch.empty_like(base_w)
    dbs = torch.empty_like(base_scale)
    dlw = [torch.empty_like(t) for t in level_w]
    dls = [torch.empty_like(t) for t in level_scale]
    dbb = torch.empty_like(base_scale) if need_dbias else None
    _check(wtconv_backward(desc, x.data_ptr(), dy.data_ptr(), base_w.data_ptr(), base_scale.data_ptr(),
                           bias.data_ptr() if bias is not None else None,
                           [t.data_ptr() for t in level_w], [t.data_ptr() for t in level_scale],
                           dx.data_ptr() if dx is not None else None, dbw.data_ptr(), dbs.data_ptr(),
                           dbb.data_ptr() if dbb is not None else None,
                           [t.data_ptr() for t in dlw], [t.data_ptr() for t in dls], workspace.data_ptr(),
                           nbytes, _stream(x.device)))
    if need_dbias:
        return dx, dbw, dbs, dlw, dls, dbb
    return dx, dbw, dbs, dlw, dls


def backward_data(dy, base_w, base_scale, level_w, level_scale, out=None, workspace=None):
    """dx alone (wtconv_backward_data): the forward pass on dy with rotated kernels."""
    import torch
    B, C, H, W, k, L = validate(dy, base_w, base_scale, level_w, level_scale, out=out)
    desc = make_desc(B, C, H, W, k, L, _dtype_code(dy))
    dx = torch.empty_like(dy) if out is None else out
    nbytes = wtconv_backward_data_workspace_bytes(desc)
    ws_ptr = None
    if nbytes:
        if not _workspace_ok(workspace, nbytes, dy.device):
            workspace = torch.empty(nbytes, dtype=torch.uint8, device=dy.device)
        ws_ptr = workspace.data_ptr()
    _check(wtconv_backward_data(desc, dy.data_ptr(), base_w.data_ptr(), base_scale.data_ptr(),
                                [t.data_ptr() for t in level_w], [t.data_ptr() for t in level_scale], dx.data_ptr(),
                                ws_ptr, nbytes, _stream(dy.device)))
    return dx


class Forward:
    """Prepared forward of one problem shape for loops that call it many times
    (serving, benchmarks): the parameters are validated once and their
    pointer arrays and the workspace are built once; `run(x, y)` checks that
    x and y match the prepared shape, dtype and device and calls
    wtconv_forward on the current stream. The parameters are kept by
    reference: later in-place updates to them are seen by later calls."""

    def __init__(self, x, base_w, base_scale, level_w, level_scale, bias=None):
        import torch
        B, C, H, W, k, L = validate(x, base_w, base_scale, level_w, level_scale, bias=bias)
        self.desc = make_desc(B, C, H, W, k, L, _dtype_code(x))
        self.x_like = (tuple(x.shape), x.dtype, x.device)
        self.nbytes = wtconv_forward_workspace_bytes(self.desc)
        self.workspace = torch.empty(self.nbytes, dtype=torch.uint8, device=x.device) if self.nbytes else None
        self.params = (base_w, base_scale, list(level_w), list(level_scale), bias)
        self.device = x.device
        self._fn = load().wtconv_forward
        self._desc_ref = ctypes.byref(self.desc)
        self._lw = _ptr_array([t.data_ptr() for t in level_w])
        self._ls = _ptr_array([t.data_ptr() for t in level_scale])
        self._bw, self._bs = base_w.data_ptr(), base_scale.data_ptr()
        self._bias = bias.data_ptr() if bias is not None else None
        self._ws = self.workspace.data_ptr() if self.workspace is not None else None
        self._nbytes = ctypes.c_size_t(self.nbytes)

    def run(self, x, y):
        """y = WTConv(x) into the preallocated `y`."""
        shape, dtype, device = self.x_like
        _require(x, "x", dtype, shape, device)
        _require(y, "y", dtype, shape, device)
        _check(self._fn(self._desc_ref, x.data_ptr(), self._bw, self._bs, self._bias, self._lw, self._ls,
                        y.data_ptr(), self._ws, self._nbytes, _stream(self.device)))
        return y


class Backward:
    """Preallocated backward of one problem: whole (wtconv_backward, `run`) or
    in its two phases (used by the benchmark to time the passes separately)."""

    def __init__(self, x, base_w, base_scale, level_w, level_scale, need_dx=True):
        import torch
        B, C, H, W, k, L = validate(x, base_w, base_scale, level_w, level_scale)
        self.desc = make_desc(B, C, H, W, k, L, _dtype_code(x))
        self.x_like = (tuple(x.shape), x.dtype, x.device)
        self.nbytes = wtconv_backward_workspace_bytes(self.desc)
        if self.nbytes == 0:
            raise WTConvError(8, "no backward plan for this shape")
        self.workspace = torch.empty(self.nbytes, dtype=torch.uint8, device=x.device)
        self.params = (base_w, base_scale, list(level_w), list(level_scale))
        self.dx = torch.empty_like(x) if need_dx else None
        self.dbw = torch.empty_like(base_w)
        self.dbs = torch.empty_like(base_scale)
        self.dlw = [torch.empty_like(t) for t in level_w]
        self.dls = [torch.empty_like(t) for t in level_scale]
        self._lw = [t.data_ptr() for t in level_w]
        self._ls = [t.data_ptr() for t in level_scale]
        self._dlw = [t.data_ptr() for t in self.dlw]
        self._dls = [t.data_ptr() for t in self.dls]
        self.device = x.device
        self.data_nbytes = wtconv_backward_data_workspace_bytes(self.desc)
        self.data_workspace = None
        # the whole call's fixed arguments, marshalled once for run()
        self._run_fn = load().wtconv_backward
        self._run_fixed = (ctypes.byref(self.desc), base_w.data_ptr(), base_scale.data_ptr(), None,
                           _ptr_array(self._lw), _ptr_array(self._ls))
        self._run_grads = (self.dbw.data_ptr(), self.dbs.data_ptr(), None, _ptr_array(self._dlw),
                           _ptr_array(self._dls), self.workspace.data_ptr(), ctypes.c_size_t(self.nbytes))

    def _check_act(self, name, t):
        shape, dtype, device = self.x_like
        _require(t, name, dtype, shape, device)

    def run(self, x, dy, dx=None):
        """wtconv_backward into the preallocated gradients; dx into `dx`, else
        into the preallocated buffer when the object was made with need_dx,
        else skipped."""
        out = dx if dx is not None else self.dx
        for name, t in (("x", x), ("dy", dy), ("dx", out)):
            if t is not None:
                self._check_act(name, t)
        desc, bw, bs, bias, lw, ls = self._run_fixed
        _check(self._run_fn(desc, x.data_ptr(), dy.data_ptr(), bw, bs, bias, lw, ls,
                            out.data_ptr() if out is not None else None, *self._run_grads, _stream(self.device)))

    def partials(self, x, dy, dx=None):
        """Writes dx into `dx`, else into the preallocated buffer when the
        object was made with need_dx, else skips it."""
        bw, bs, _, _ = self.params
        out = dx if dx is not None else self.dx
        for name, t in (("x", x), ("dy", dy), ("dx", out)):
            if t is not None:
                self._check_act(name, t)
        _check(wtconv_backward_partials(self.desc, x.data_ptr(), dy.data_ptr(), bw.data_ptr(), bs.data_ptr(),
                                        self._lw, self._ls, out.data_ptr() if out is not None else None,
                                        self.workspace.data_ptr(), self.nbytes, _stream(self.device)))

    def data(self, dy, dx):
        """dx alone (wtconv_backward_data) into `dx`."""
        bw, bs, _, _ = self.params
        self._check_act("dy", dy)
        self._check_act("dx", dx)
        if self.data_nbytes and self.data_workspace is None:
            import torch
            self.data_workspace = torch.empty(self.data_nbytes, dtype=torch.uint8, device=self.device)
        _check(wtconv_backward_data(self.desc, dy.data_ptr(), bw.data_ptr(), bs.data_ptr(), self._lw, self._ls,
                                    dx.data_ptr(),
                                    self.data_workspace.data_ptr() if self.data_workspace is not None else None,
                                    self.data_nbytes, _stream(self.device)))

    def finalize(self):
        bw, bs, _, _ = self.params
        _check(wtconv_backward_finalize(self.desc, bw.data_ptr(), bs.data_ptr(), None, self._lw, self._ls,
                                        self.dbw.data_ptr(), self.dbs.data_ptr(), None, self._dlw, self._dls,
                                        self.workspace.data_ptr(), self.nbytes, _stream(self.device)))
