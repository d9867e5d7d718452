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
    8: "WTCONV_ERR_UNSUPPORTED", 9: "WTCONV_ERR_HIP",
}
EXPORTS = ["wtconv_forward_workspace_bytes", "wtconv_forward", "wtconv_backward", "wtconv_backward_workspace_bytes",
           "wtconv_backward_partials", "wtconv_backward_finalize", "wtconv_backward_data_workspace_bytes",
           "wtconv_backward_data", "wtconv_status_string", "wtconv_version"]
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
    level_* are lists of addresses."""
    return load().wtconv_forward(ctypes.byref(desc), x, base_w, base_scale, base_bias, _ptr_array(level_w),
                                 _ptr_array(level_scale), y, workspace, ctypes.c_size_t(workspace_bytes), stream)


def wtconv_backward_workspace_bytes(desc: Desc) -> int:
    return int(load().wtconv_backward_workspace_bytes(ctypes.byref(desc)))


def wtconv_backward(desc: Desc, x, dy, base_w, base_scale, base_bias, level_w, level_scale, dx, d_base_w,
                    d_base_scale, d_base_bias, d_level_w, d_level_scale, workspace, workspace_bytes, stream) -> int:
    return load().wtconv_backward(ctypes.byref(desc), x, dy, base_w, base_scale, base_bias, _ptr_array(level_w),
                                  _ptr_array(level_scale), dx, d_base_w, d_base_scale, d_base_bias,
                                  _ptr_array(d_level_w), _ptr_array(d_level_scale), workspace,
                                  ctypes.c_size_t(workspace_bytes), stream)


def wtconv_backward_partials(desc: Desc, x, dy, base_w, base_scale, level_w, level_scale, dx, workspace,
                             workspace_bytes, stream) -> int:
    return load().wtconv_backward_partials(ctypes.byref(desc), x, dy, base_w, base_scale, _ptr_array(level_w),
                                           _ptr_array(level_scale), dx, workspace,
                                           ctypes.c_size_t(workspace_bytes), stream)


def wtconv_backward_finalize(desc: Desc, base_w, base_scale, base_bias, level_w, level_scale, d_base_w,
                             d_base_scale, d_base_bias, d_level_w, d_level_scale, workspace, workspace_bytes,
                             stream) -> int:
    return load().wtconv_backward_finalize(ctypes.byref(desc), base_w, base_scale, base_bias, _ptr_array(level_w),
                                           _ptr_array(level_scale), d_base_w, d_base_scale, d_base_bias,
                                           _ptr_array(d_level_w), _ptr_array(d_level_scale), workspace,
                                           ctypes.c_size_t(workspace_bytes), stream)


def wtconv_backward_data_workspace_bytes(desc: Desc) -> int:
    return int(load().wtconv_backward_data_workspace_bytes(ctypes.byref(desc)))


def wtconv_backward_data(desc: Desc, dy, base_w, base_scale, level_w, level_scale, dx, workspace, workspace_bytes,
                         stream) -> int:
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


def _require(t, name, dtype=None):
    import torch
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise ValueError(f"{name} must be a GPU tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")


def _stream(device):
    import torch
    return torch.cuda.current_stream(device).cuda_stream


def forward(x, base_w, base_scale, level_w, level_scale, out=None, workspace=None, bias=None):
    """y = WTConv(x) on the current stream. x: [B,C,H,W] fp32/bf16/fp16 on the GPU;
    base_w [C,k,k], base_scale [C], level_w list of [4C,k,k], level_scale list of [4C] (fp32);
    bias: the base bias [C] (fp32) or None.
    Large planes need a device workspace; one is allocated if `workspace` is None or too small."""
    import torch
    _require(x, "x")
    B, C, H, W = x.shape
    k = base_w.shape[-1]
    L = len(level_w)
    for name, t in [("base_w", base_w), ("base_scale", base_scale)] + \
            [(f"level_w[{i}]", t) for i, t in enumerate(level_w)] + \
            [(f"level_scale[{i}]", t) for i, t in enumerate(level_scale)] + \
            ([("bias", bias)] if bias is not None else []):
        _require(t, name, torch.float32)
    y = torch.empty_like(x) if out is None else out
    desc = make_desc(B, C, H, W, k, L, _dtype_code(x))
    nbytes = wtconv_forward_workspace_bytes(desc)
    ws_ptr = None
    if nbytes:
        if workspace is None or workspace.numel() * workspace.element_size() < nbytes:
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
    _require(x, "x")
    _require(dy, "dy", x.dtype)
    B, C, H, W = x.shape
    k = base_w.shape[-1]
    L = len(level_w)
    desc = make_desc(B, C, H, W, k, L, _dtype_code(x))
    nbytes = wtconv_backward_workspace_bytes(desc)
    if nbytes == 0:
        raise WTConvError(8, "no backward plan for this shape")
    if workspace is None or workspace.numel() * workspace.element_size() < nbytes:
        workspace = torch.empty(nbytes, dtype=torch.uint8, device=x.device)
    dx = torch.empty_like(x) if need_dx else None
    dbw = torch.empty_like(base_w)
    dbs = torch.empty_like(base_scale)
    dlw = [torch.empty_like(t) for t in level_w]
    dls = [torch.empty_like(t) for t in level_scale]
    dbb = torch.empty_like(base_scale) if need_dbias else None
    if bias is not None:
        _require(bias, "bias", torch.float32)
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
    _require(dy, "dy")
    B, C, H, W = dy.shape
    desc = make_desc(B, C, H, W, base_w.shape[-1], len(level_w), _dtype_code(dy))
    dx = torch.empty_like(dy) if out is None else out
    nbytes = wtconv_backward_data_workspace_bytes(desc)
    ws_ptr = None
    if nbytes:
        if workspace is None or workspace.numel() * workspace.element_size() < nbytes:
            workspace = torch.empty(nbytes, dtype=torch.uint8, device=dy.device)
        ws_ptr = workspace.data_ptr()
    _check(wtconv_backward_data(desc, dy.data_ptr(), base_w.data_ptr(), base_scale.data_ptr(),
                                [t.data_ptr() for t in level_w], [t.data_ptr() for t in level_scale], dx.data_ptr(),
                                ws_ptr, nbytes, _stream(dy.device)))
    return dx


class Backward:
    """Preallocated backward of one problem, callable in its two phases
    (used by the benchmark to time the fused pass and the finalize separately)."""

    def __init__(self, x, base_w, base_scale, level_w, level_scale, need_dx=True):
        import torch
        B, C, H, W = x.shape
        self.desc = make_desc(B, C, H, W, base_w.shape[-1], len(level_w), _dtype_code(x))
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

    def partials(self, x, dy, dx=None):
        bw, bs, _, _ = self.params
        out = dx if dx is not None else self.dx
        _check(wtconv_backward_partials(self.desc, x.data_ptr(), dy.data_ptr(), bw.data_ptr(), bs.data_ptr(),
                                        self._lw, self._ls, out.data_ptr() if out is not None else None,
                                        self.workspace.data_ptr(), self.nbytes, _stream(self.device)))

    def data(self, dy, dx):
        """dx alone (wtconv_backward_data) into `dx`."""
        bw, bs, _, _ = self.params
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
