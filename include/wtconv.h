/*
 * wtconv.h -- C ABI of the MI355X (gfx950) fused WTConv library, libwtconv.so.
 *
 * The operator (Aflalo et al., Section 2.1, Algorithm 1) maps an input
 * x[B][C][H][W] to y[B][C][H][W]:
 *
 *   y = s0 * (x (*) W0 + b0) + R,  R = sum over levels l = 1..L of the Haar
 *                                      synthesis of Z_l,
 *   Z_l = s_l * (Y_l (*) W_l),   Y_l = one orthonormal 2x2 Haar analysis
 *                                    level applied to the raw LL band of
 *                                    level l-1 (Y_1 from x),
 *
 * where (*) is the depthwise k x k "same" cross-correlation with zero padding
 * (PyTorch conv2d semantics), W0 is one k x k kernel per channel, W_l one
 * k x k kernel per subband channel (4C of them), s0 one scale per channel,
 * b0 one bias per channel (the base bias of Algorithm 1, optional: NULL means
 * zero) and s_l one scale per subband channel.
 * Odd H or W are zero-padded at the bottom/right before each analysis level
 * and cropped after synthesis, which is the same as zero-extending x: level l
 * lives on a ceil(H/2^l) x ceil(W/2^l) grid.
 *
 * Subband channel layout: row 4c+q of a level's [4C][k][k] kernel and [4C]
 * scale belongs to channel c, band q = 0 LL, 1 LH, 2 HL, 3 HH, with the band
 * formulas of eq. (butterfly), Section 4.1, on the patch [[a,b],[c,d]]:
 * LL=(a+b+c+d)/2, LH=(a+b-c-d)/2, HL=(a-b+c-d)/2, HH=(a-b-c+d)/2.
 *
 * The kernels compute the operator in one pass per plane with the three
 * reformulations of Section 4: Haar analysis recomputed on chip (Section
 * 4.1), the bit-indexed closed-form synthesis of Proposition 2 (Section 4.2),
 * and the scales folded into the kernels and the bias (eq. fold, Section 4.3).
 * The backward pass recovers the unfolded parameter gradients with
 * eq. (foldgrad).
 *
 * Conventions common to all entry points:
 *   - Tensors are NCHW-contiguous device pointers. x, y, dy and dx have the
 *     element type given by desc->dtype; kernels, scales and all parameter
 *     gradients are float32. Accumulation is float32 for every dtype; bf16 and
 *     fp16 results are rounded to nearest even.
 *   - level_w / level_scale (and their gradients) are HOST arrays of L DEVICE
 *     pointers: level_w[l-1] -> [4C][k][k], level_scale[l-1] -> [4C].
 *   - The caller owns every buffer. The library allocates no device memory;
 *     scratch space comes from a caller-provided workspace (or, for
 *     wtconv_backward_noalloc, from a static device array in the library).
 *   - Work is enqueued on `stream` and is asynchronous. Argument errors are
 *     detected on the host before any HIP call and returned synchronously;
 *     launch errors are returned as WTCONV_ERR_HIP; device faults surface at
 *     the caller's next synchronisation.
 *   - Gradient outputs are overwritten, not accumulated into.
 *   - Entry points are reentrant and thread-safe; the library's global state
 *     is the static scratch of wtconv_backward_noalloc (see there) and a
 *     mutex-guarded cache of execution plans by descriptor (64 entries, a
 *     plan depends only on the descriptor). Results are bitwise reproducible
 *     for identical inputs and shapes.
 *   - Supported: B, C, H, W >= 1; odd k with 1 <= k <= 9; 0 <= L <= 8. Even
 *     k has no centred halo (Section 4.1 takes the radius (k-1)/2) and is
 *     refused. The paper's experiments take k = 3, 5 and 7; k = 9 runs the same
 *     kernels, whose per-lane kernel-gradient sums then overflow the register
 *     budget the backward kernels are sized for (it is correct, not tuned).
 *     Planes whose
 *     fused working set fits one compute unit's 160 KB of LDS (float32, k = 5:
 *     forward up to about 120 x 120 pixels, backward up to about 112 x 112, or
 *     about 90 x 90 at L = 1) run
 *     in one pass; larger planes use a split with a workspace.
 */
#ifndef WTCONV_H
#define WTCONV_H

#include <stddef.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define WTCONV_MAX_LEVELS 8
#define WTCONV_MAX_KSIZE 9

typedef enum {
    WTCONV_F32 = 0,
    WTCONV_BF16 = 1,
    WTCONV_F16 = 2
} wtconv_dtype;

typedef enum {
    WTCONV_OK = 0,
    WTCONV_ERR_NULL = 1,        /* a required pointer is NULL                     */
    WTCONV_ERR_SHAPE = 2,       /* B, C, H or W < 1, or a size overflows int      */
    WTCONV_ERR_KSIZE = 3,       /* k even, k < 1 or k > 9                         */
    WTCONV_ERR_LEVELS = 4,      /* L < 0 or L > WTCONV_MAX_LEVELS                 */
    WTCONV_ERR_DTYPE = 5,       /* unknown dtype                                  */
    WTCONV_ERR_ALIAS = 6,       /* an output overlaps an input or another output  */
    WTCONV_ERR_WORKSPACE = 7,   /* workspace NULL or smaller than required        */
    WTCONV_ERR_UNSUPPORTED = 8, /* no execution plan for this shape               */
    WTCONV_ERR_HIP = 9,         /* a HIP runtime call or kernel launch failed     */
    WTCONV_ERR_SCRATCH = 10     /* wtconv_backward_noalloc: the problem needs more
                                   workspace than WTCONV_NOALLOC_SCRATCH_BYTES     */
} wtconv_status;

/* Problem descriptor (host memory). */
typedef struct {
    int B, C, H, W; /* batch, channels, height, width                               */
    int k;          /* kernel size (odd), radius (k-1)/2                             */
    int L;          /* Haar levels; L = 0 gives y = s0 * (x (*) W0)                 */
    wtconv_dtype dtype;
} wtconv_desc;

/* Bytes of device workspace wtconv_forward needs for `desc` (0 when the planes
 * are processed on chip in one pass, or on a bad desc). */
size_t wtconv_forward_workspace_bytes(const wtconv_desc* desc);

/*
 * Forward pass, Algorithm 1 (Section 2.1).
 *   x            [B][C][H][W] dtype
 *   base_w       [C][k][k] float32           base_scale [C] float32
 *   base_bias    [C] float32, or NULL for no bias
 *   level_w      host array of L device ptrs, each [4C][k][k] float32
 *   level_scale  host array of L device ptrs, each [4C] float32
 *   y            [B][C][H][W] dtype; must not overlap any input
 *   workspace    device memory of at least wtconv_forward_workspace_bytes(desc)
 *                bytes, 16-byte aligned; may be NULL when that size is 0. Its
 *                contents are scratch.
 * level_w / level_scale may be NULL when L = 0. Planes whose working set fits
 * one compute unit's LDS are read once and written once; larger planes are
 * split (the coarse levels run on the quarter-size level-1 carrier held in the
 * workspace, the base path and level 1 run on tiles with a halo).
 */
wtconv_status wtconv_forward(const wtconv_desc* desc, const void* x, const float* base_w,
                             const float* base_scale, const float* base_bias, const float* const* level_w,
                             const float* const* level_scale, void* y, void* workspace,
                             size_t workspace_bytes, hipStream_t stream);

/* Bytes of device workspace wtconv_backward needs for `desc` (0 on a bad desc). */
size_t wtconv_backward_workspace_bytes(const wtconv_desc* desc);

/*
 * Backward pass: gradients of sum(y * dy) with respect to x and every
 * parameter (Section 2.2 for the Haar steps, eq. foldgrad of Section 4.3 for
 * the folded scales and bias).
 *   x, dy              [B][C][H][W] dtype
 *   base_bias          [C] float32 or NULL (zero): it enters d_base_scale
 *                      (d s0 = <G0, W0> + b0 * sum(dy))
 *   dx                 [B][C][H][W] dtype, or NULL to skip the input gradient
 *   d_base_w [C][k][k], d_base_scale [C]                           float32
 *   d_base_bias [C] float32 (s0 * sum(dy) per channel), or NULL to skip it
 *   d_level_w / d_level_scale: host arrays of L device ptrs, [4C][k][k] / [4C]
 *   workspace          device memory of at least
 *                      wtconv_backward_workspace_bytes(desc) bytes (16-byte
 *                      aligned); its contents are scratch
 * Outputs must not overlap the inputs, each other or the workspace.
 * For planes above 16 x 16 with L >= 1, and planes above 8 x 8 with L = 1 or
 * 2 (any L for k = 7, and for k = 5 up to 12 x 12), dx is the forward pass on
 * dy with every kernel rotated by 180 degrees (the adjoint of the operator)
 * and the kernel gradients come from a separate correlation pass over x and
 * dy; the final reduction of those gradients then runs in the launch that
 * forms dx (wtconv_backward_partials followed by wtconv_backward_finalize
 * launch it on its own, with bit-identical results). For other shapes one
 * fused pass per plane produces both.
 */
wtconv_status wtconv_backward(const wtconv_desc* desc, const void* x, const void* dy,
                              const float* base_w, const float* base_scale, const float* base_bias,
                              const float* const* level_w, const float* const* level_scale,
                              void* dx, float* d_base_w, float* d_base_scale, float* d_base_bias,
                              float* const* d_level_w, float* const* d_level_scale,
                              void* workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * The two phases of wtconv_backward, for callers that want to schedule them
 * separately (wtconv_backward is exactly partials followed by finalize).
 *
 * wtconv_backward_partials: the passes over every plane. Writes dx (if
 *   dx != NULL) and per-workgroup kernel-gradient partial sums (and the sum
 *   of dy per channel) into `workspace`. The bias does not enter this phase;
 *   otherwise the same arguments and checks as wtconv_backward.
 * wtconv_backward_finalize: sums the partials of `workspace` in a fixed order
 *   and unfolds them into the parameter gradients (eq. foldgrad): d_base_w =
 *   s0 * G0, d_base_scale = <G0, W0> + b0 * sum(dy), d_base_bias = s0 *
 *   sum(dy) (if not NULL), and d_level_w = s_l * G_l, d_level_scale =
 *   <G_l, W_l> per subband channel of every level. `workspace` must hold the
 *   partials of a preceding
 *   wtconv_backward_partials call with the same descriptor and parameters,
 *   enqueued earlier on the same stream (or otherwise ordered before it).
 */
wtconv_status wtconv_backward_partials(const wtconv_desc* desc, const void* x, const void* dy,
                                       const float* base_w, const float* base_scale,
                                       const float* const* level_w, const float* const* level_scale,
                                       void* dx, void* workspace, size_t workspace_bytes,
                                       hipStream_t stream);

wtconv_status wtconv_backward_finalize(const wtconv_desc* desc, const float* base_w, const float* base_scale,
                                       const float* base_bias, const float* const* level_w,
                                       const float* const* level_scale, float* d_base_w, float* d_base_scale,
                                       float* d_base_bias, float* const* d_level_w, float* const* d_level_scale,
                                       const void* workspace, size_t workspace_bytes, hipStream_t stream);

/* Bytes of device workspace wtconv_backward_data needs for `desc` (the same as
 * the forward pass; 0 when the planes are processed on chip, or on a bad desc). */
size_t wtconv_backward_data_workspace_bytes(const wtconv_desc* desc);

/*
 * Input gradient only: dx = d sum(y * dy) / dx. The operator is linear in x
 * and its adjoint is the same operator with every kernel rotated by 180
 * degrees (the adjoint of a "same" correlation is the correlation with the
 * rotated kernel; Haar synthesis and analysis are each other's transposes,
 * Proposition 1), so this is the forward pass on dy with rotated kernels and
 * no bias. For callers that do not need parameter gradients, or that schedule
 * the input gradient separately from wtconv_backward_partials(dx = NULL) and
 * wtconv_backward_finalize.
 *   dy           [B][C][H][W] dtype
 *   base_w, base_scale, level_w, level_scale: as for wtconv_forward
 *   dx           [B][C][H][W] dtype; must not overlap any input
 *   workspace    at least wtconv_backward_data_workspace_bytes(desc) bytes,
 *                16-byte aligned (may be NULL when that size is 0)
 */
wtconv_status wtconv_backward_data(const wtconv_desc* desc, const void* dy, const float* base_w,
                                   const float* base_scale, const float* const* level_w,
                                   const float* const* level_scale, void* dx, void* workspace,
                                   size_t workspace_bytes, hipStream_t stream);

/*
 * wtconv_backward without a workspace argument, for callers that cannot
 * allocate device memory: code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation. Same arguments, checks, kernels and
 * results as wtconv_backward; the workspace is a static device array of
 * WTCONV_NOALLOC_SCRATCH_BYTES inside the library (one per GPU it runs on,
 * held until the process ends), so the call allocates nothing.
 *   Returns WTCONV_ERR_SCRATCH, before any HIP call, when
 *   wtconv_backward_workspace_bytes(desc) exceeds that size (it covers every
 *   ConvNeXt-T stage shape at B = 128, L <= 5; large planes split into
 *   carriers and exceed it).
 *   The array is shared by every call on one GPU and keeps the last call's
 *   contents (each call overwrites what it reads): calls that overlap on one
 *   GPU, e.g. on two streams at once, race and must be ordered by the caller.
 *   The device is the one `stream` belongs to; the array's address there is
 *   looked up on the first call on that device.
 */
#define WTCONV_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)

wtconv_status wtconv_backward_noalloc(const wtconv_desc* desc, const void* x, const void* dy,
                                      const float* base_w, const float* base_scale, const float* base_bias,
                                      const float* const* level_w, const float* const* level_scale,
                                      void* dx, float* d_base_w, float* d_base_scale, float* d_base_bias,
                                      float* const* d_level_w, float* const* d_level_scale,
                                      hipStream_t stream);

/* Static, human-readable name of a status code. */
const char* wtconv_status_string(wtconv_status status);

/* Library ABI version (major * 10000 + minor * 100 + patch). */
int wtconv_version(void);

#ifdef __cplusplus
}
#endif

#endif /* WTCONV_H */
