"""I/O, arithmetic and roofline accounting for the WTConv operator.

Closed forms from the paper:
  * eq. (qref), Section 3.1: reference traffic 7N + 43/3 N (1 - 4^-L) elements;
  * eq. (mac), Section 3.2: N [k^2 + (k^2 + 8) 4/3 (1 - 4^-L)] multiply-accumulates;
  * eq. (qfused), Section 4.4: fused multi-pass traffic
    4N + 13/3 N (1 - 4^-L) - N 4^-L elements, and eq. (qratio) their ratio.

Plus the accounting of the single-pass design in this library, which reads
every activation once and writes every result once:
  * forward: x read, y written                      -> 2N elements;
  * backward: x and dy read, dx written             -> 3N elements;
  * plus the fp32 parameters (and parameter gradients) once.
Arithmetic of the single-pass design counts only what the method must do:
k^2 FMAs per output pixel of the base convolution and per subband
coefficient of every level, on the exact ceil(H/2^l) x ceil(W/2^l) grids.

MI355X peaks used for rooflines: HBM3E 8.0 TB/s; 256 compute units at
2.4 GHz, each retiring 64 fp32 FMA lanes per clock without packed-FP32
instructions (78.6 TFLOP/s, 39.3 T FMA/s); the 157.3 TFLOP/s vector figure
assumes packed FP32 FMA, which this library does not emit.
"""
from dataclasses import dataclass

HBM_PEAK_GBPS = 8000.0
CUS = 256
CLOCK_HZ = 2.4e9
LANES_PER_CU = 64
FP32_FMA_PER_S = CUS * LANES_PER_CU * CLOCK_HZ          # 39.32e12 FMA/s (non-packed)
FP32_FLOPS = 2.0 * FP32_FMA_PER_S                      # 78.6 TFLOP/s
FP32_FLOPS_PACKED = 2.0 * FP32_FLOPS                   # 157.3 TFLOP/s (packed FP32, not used)


def q_ref(L: int) -> float:
    """Reference-implementation traffic per forward, in units of N elements (eq. qref)."""
    return 7.0 + 43.0 / 3.0 * (1.0 - 4.0 ** (-L))


def q_fused(L: int) -> float:
    """The paper's fused multi-pass traffic per forward, in units of N (eq. qfused)."""
    return 4.0 + 13.0 / 3.0 * (1.0 - 4.0 ** (-L)) - 4.0 ** (-L)


def q_ratio(L: int) -> float:
    """eq. (qratio)."""
    return q_ref(L) / q_fused(L)


def mac_ref(k: int, L: int) -> float:
    """Reference multiply-accumulates per input element (eq. mac)."""
    return k * k + (k * k + 8) * 4.0 / 3.0 * (1.0 - 4.0 ** (-L))


def level_grid(H: int, W: int, l: int):
    for _ in range(l):
        H, W = (H + 1) // 2, (W + 1) // 2
    return H, W


def coef_sites(H: int, W: int, L: int) -> int:
    """Subband coefficients per plane over levels 1..L (4 bands per site)."""
    n = 0
    for l in range(1, L + 1):
        h, w = level_grid(H, W, l)
        n += 4 * h * w
    return n


def param_count(C: int, k: int, L: int) -> int:
    """fp32 parameters: base kernel + base scale + L x (4C kernels + 4C scales)."""
    return C * (k * k + 1) + L * 4 * C * (k * k + 1)


@dataclass
class Work:
    bytes_fwd: float
    bytes_bwd: float
    fma_fwd: float
    fma_bwd: float

    @property
    def bytes_fwdbwd(self) -> float:
        return self.bytes_fwd + self.bytes_bwd

    @property
    def fma_fwdbwd(self) -> float:
        return self.fma_fwd + self.fma_bwd


def elem_bytes(dtype: str) -> int:
    return {"f32": 4, "bf16": 2, "f16": 2}[dtype]


def single_pass_work(B: int, C: int, H: int, W: int, k: int, L: int, dtype: str) -> Work:
    """Algorithmic bytes and FMAs of the single-pass forward and backward."""
    N = B * C * H * W
    e = elem_bytes(dtype)
    P = param_count(C, k, L)
    coefs = B * C * coef_sites(H, W, L)
    fma_fwd = k * k * (N + coefs)
    # backward: dX has the forward's structure; the kernel gradients add one
    # correlation (k^2 FMAs) per pixel and per coefficient.
    fma_bwd = 2 * k * k * (N + coefs)
    return Work(
        bytes_fwd=2.0 * N * e + 4.0 * P,
        bytes_bwd=3.0 * N * e + 4.0 * P + 4.0 * P,
        fma_fwd=float(fma_fwd),
        fma_bwd=float(fma_bwd),
    )


def hbm_floor_s(nbytes: float) -> float:
    return nbytes / (HBM_PEAK_GBPS * 1e9)


def fma_floor_s(fma: float) -> float:
    return fma / FP32_FMA_PER_S
