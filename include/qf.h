/*
 * qf.h -- C ABI of libqf: deployment-aligned simulated ("fake") quantization and the
 * quantization-aware linear layer with a straight-through backward, for AMD MI355X (gfx950).
 *
 * Method: QATFactory, Sec. 3.2 "Deployment-aligned simulated quantization".
 *   Q(X) -> (C, theta), Q^-1(C, theta) -> X_hat                         Eq. quantize-dequantize
 *   W_hat = Q^-1(Q(W)), A_hat = Q^-1(Q(A)), O = W_hat A_hat              Eq. fakequant
 *   dL/dW ~= dL/dO A_hat^T                                               Eq. ste
 *   dL/dA ~= W_hat^T dL/dO                                               Eq. activation-ste
 * Formats (Sec. 3.2.3, Tab. formats): NVFP4 (E2M1 + E4M3 per 16 + FP32 tensor scale),
 * MXFP4 (E2M1 + E8M0 per 32), Q4_K (uint4 + 6-bit scales/mins per 32 + FP16 per 256).
 *
 * Conventions (all entry points)
 *  - Tensors are row-major.  Activations are [M, K] (tokens x in-features), weights follow
 *    nn.Linear: [N, K] (out x in), outputs [M, N].  Quantization blocks run along K.
 *  - bf16 / fp16 tensors are passed as raw 16-bit words (uint16_t), little-endian.
 *  - Every tensor pointer is DEVICE memory owned by the caller.  The library allocates no
 *    device memory; scratch comes from the caller's workspace (qf_workspace_size).
 *  - Calls are asynchronous on `stream` (a hipStream_t; 0 = the null stream).  Inputs must
 *    stay valid and outputs must not be read until the stream reaches that point.
 *  - Every call returns a qf_status.  Validation is done on the host before any launch:
 *    on error nothing is launched and qf_last_error() returns a message (thread-local).
 *    Non-finite data is never an error; it propagates as each format defines.
 *  - Alignment: every tensor base pointer must be 16-byte aligned and every leading
 *    dimension a multiple of 8 elements (QF_EALIGN otherwise).
 *  - Nibble order: two 4-bit codes per byte, element 2i in the LOW nibble.  Code layout:
 *    bit 3 = sign, bits 0-2 = E2M1 magnitude index into {0, .5, 1, 1.5, 2, 3, 4, 6}.
 *  - Scale layout: plain row-major [R, K/block] bytes (E4M3 for NVFP4, E8M0 for MXFP4).
 */
#ifndef QF_H
#define QF_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#if defined(__GNUC__)
#define QF_API __attribute__((visibility("default")))
#else
#define QF_API
#endif

typedef void* qf_stream_t; /* a hipStream_t */

typedef enum {
    QF_OK = 0,
    QF_EINVAL = 1,   /* null required pointer, bad enum, aliasing that the call forbids */
    QF_ESHAPE = 2,   /* negative size, K not a multiple of the format's block, ld < K   */
    QF_EALIGN = 3,   /* pointer not 16-byte aligned or ld not a multiple of 8          */
    QF_ENOTSUP = 4,  /* valid request that the library does not implement             */
    QF_EDEVICE = 5   /* a HIP launch failed (message carries the HIP error string)      */
} qf_status;

typedef enum {
    QF_FMT_NONE = 0,   /* no quantization: the tensor is used as is (W4A16 activations)  */
    QF_FMT_NVFP4 = 1,
    QF_FMT_MXFP4 = 2,
    QF_FMT_Q4K = 3     /* weights only (Tab. formats: W4A16)                              */
} qf_format;

typedef enum {
    QF_AMAX_COMPUTE = 0, /* the call computes g = max|x| and stores it in *amax             */
    QF_AMAX_GIVEN = 1    /* *amax already holds g (running activation amax, Sec. 3.2.3
                            NVFP4 paragraph; or a tied-group max, "Engine-specific scale
                            sharing")                                                    */
} qf_amax_mode;

/* Library version (major*10000 + minor*100 + patch) and the last error on this thread. */
QF_API int qf_version(void);
QF_API const char* qf_last_error(void);

/*
 * qf_amax -- tensor amax g = max |x| over a bf16 [R, K] tensor (Sec. 3.2.1: scales derive
 * from the maximum absolute value).  `amax` is a device FP32 scalar.
 *   accumulate = 0: *amax = g.   accumulate = 1: *amax = max(*amax, g) -- the running
 *   activation amax of Sec. 3.2.3 (NVFP4 paragraph), and the way to build a tied-scale group
 *   ("Engine-specific scale sharing": call once per member).
 * K may be any size (no block constraint; ldx >= K, ldx % 8 == 0): elements past K in a row
 * are never read.  NaN inputs make *amax NaN.  R = 0 or K = 0 leaves a zero (accumulate = 0)
 * or unchanged value.  One kernel dispatch (no clearing dispatch before it): the workgroups
 * fold into one of 1024 per-device reduction slots, taken in turn per pass (one per tensor of
 * a batch; grouped calls allow at most 1024 experts) and left clear by the pass's last
 * workgroups, so passes on different streams run independently unless 1024 further slots are
 * taken while one is still in flight.  Graph-capturable (no memset nodes).
 */
QF_API qf_status qf_amax(const uint16_t* x, int64_t R, int64_t K, int64_t ldx, float* amax,
                  int accumulate, qf_stream_t stream);

/*
 * qf_fakequant_nvfp4 -- NVFP4 quantize + dequantize (Eqs. nvfp4, nvfp4-dequant).
 *   x       bf16 [R, K] (row stride ldx elements), K % 16 == 0.
 *   amax    device FP32 scalar, required.  amax_mode = QF_AMAX_COMPUTE: the call writes g;
 *           QF_AMAX_GIVEN: the call reads g.
 *   s_out   device FP32 scalar or NULL: receives the tensor decode scale S = g / 2688
 *           (2688 = 6 * 448, largest E2M1 times largest E4M3).  Must not alias `amax`.
 *   codes   [R, K/2] bytes or NULL;  scales [R, K/16] E4M3 bytes or NULL;
 *   xhat    bf16 [R, K] (row stride K) or NULL.
 * Per block of 16: t = a_b / (6 S) rounded to the nearest E4M3 (saturating at 448),
 * D_b = S * s_E4M3, codes = nearest E2M1 to |x| * (1 / D_b) (ties to even, saturating),
 * x_hat = bf16(+-V * D_b).  g = 0 gives all-zero scales and codes carrying only the sign.
 */
QF_API qf_status qf_fakequant_nvfp4(const uint16_t* x, int64_t R, int64_t K, int64_t ldx,
                             float* amax, int amax_mode, float* s_out, uint8_t* codes,
                             uint8_t* scales, uint16_t* xhat, qf_stream_t stream);

/*
 * qf_fakequant_mxfp4 -- MXFP4 quantize + dequantize (Eqs. mxfp4, mxfp4-dequant).
 *   x bf16 [R, K], K % 32 == 0.  codes [R, K/2] or NULL; scales [R, K/32] E8M0 or NULL;
 *   xhat bf16 [R, K] or NULL.
 * Per block of 32: p = floor(log2 max|x|) - 2 clamped to [-127, 127] (code p + 127),
 * codes = nearest E2M1 to |x| / 2^p (ties to even, saturating at 6), x_hat = +-V * 2^p.
 * All-zero block: code 0.  Block holding Inf/NaN: scale 0xFF, codes 0, x_hat NaN (0x7FC0).
 */
QF_API qf_status qf_fakequant_mxfp4(const uint16_t* x, int64_t R, int64_t K, int64_t ldx,
                             uint8_t* codes, uint8_t* scales, uint16_t* xhat,
                             qf_stream_t stream);

/*
 * qf_fakequant_q4k -- Q4_K quantize + dequantize + llama.cpp block packing
 * (Eqs. q4k, q4k-dequant; Sec. 3.5 engine-native export).
 *   x bf16 [R, K], K % 256 == 0.  packed [R, K/256, 144] bytes or NULL; xhat bf16 [R, K] or NULL.
 * Block of 144 bytes: FP16 d, FP16 dmin, 12 bytes of 6-bit scales/mins, 128 bytes of codes
 * (byte 32c+l: code 64c+l in the low nibble, code 64c+32+l in the high nibble).
 * Scale search ("min-max"): per sub-block of 32 the range [min(0, min x), max x] is split
 * into 15 steps; d, dmin = FP16(max step / 63), FP16(max offset / 63); 6-bit scale and min =
 * nearest integers; code = nearest integer to (x + dmin*m6) / (d*s6) clamped to [0, 15];
 * x_hat = bf16(d*s6*code - dmin*m6).  Signed zeros in x count as +0.
 */
QF_API qf_status qf_fakequant_q4k(const uint16_t* x, int64_t R, int64_t K, int64_t ldx,
                           uint8_t* packed, uint16_t* xhat, qf_stream_t stream);

/*
 * qf_fakequant_q4k_mse -- Q4_K (same 144-byte blocks and x_hat convention as qf_fakequant_q4k)
 * whose sub-block steps and offsets come from a search minimizing ||x - x_hat||^2, the
 * objective of the Q4_K post-training baseline (Sec. 4 "Quantization-aware distillation":
 * scales that minimize ||W - W_q||^2).  The search is this library's own: per sub-block of 32,
 * 17 candidate steps (hi - lo) / (14 + k/4) (lo = min(0, min x), hi = max x) each give codes,
 * to which step and offset are refitted by least squares (offset >= 0); the candidate with
 * the smallest squared error wins.  Each super-block keeps the searched result or the
 * min-max one (qf_fakequant_q4k), whichever decodes with the smaller error, so it is never
 * worse.  FP32 sums over a sub-block: per 8 consecutive elements in order, then
 * (g0 + g1) + (g2 + g3); over a super-block: ((s0 + s1) + (s2 + s3)) + ((s4 + s5) + (s6 + s7)).
 *   x bf16 [R, K], K % 256 == 0; packed [R, K/256, 144] or NULL; xhat bf16 [R, K] or NULL.
 */
QF_API qf_status qf_fakequant_q4k_mse(const uint16_t* x, int64_t R, int64_t K, int64_t ldx,
                                      uint8_t* packed, uint16_t* xhat, qf_stream_t stream);

/* ---------------------------------------------------------------------------------------
 * Quantization-aware linear layer (Eqs. fakequant, ste, activation-ste)
 * ------------------------------------------------------------------------------------ */

/* flags */
#define QF_FLAG_REUSE_WS 1u /* the caller keeps the workspace from the forward to the backward
                               (same X, W, desc and flags).  The forward then also writes A_hat^T
                               (X^T for unquantized activations) into it from the A tiles its
                               GEMM stages (M % 8 == 0, N <= 8192), and the backward takes dW's
                               operand from there instead of transposing or quantizing X; without a
                               saved buffer it also takes the packed W_hat and A_hat from the
                               workspace.  The bits are identical either way */
#define QF_FLAG_DECODE_IN_GEMM 2u /* forward: decode the packed weight inside the GEMM's
                               prologue instead of writing W_hat in bf16 to the workspace and
                               running a plain bf16 GEMM (identical Y; K a multiple of 64, else
                               the flag is ignored).  Not the default: on MI355X the decoded
                               tiles' LDS writes cost more than the bf16 W_hat pass saves */

typedef struct {
    int64_t M, N, K;      /* X [M, K], W [N, K], Y [M, N]                                  */
    int64_t ldx, ldw, ldy;/* row strides (elements) of X / dX, W, Y / dY; 0 means dense     */
    int32_t wfmt;         /* qf_format of the weight                                       */
    int32_t afmt;         /* qf_format of the activation (QF_FMT_NONE = W4A16 training)    */
    float* w_amax;        /* NVFP4 weight: device FP32 scalar or NULL.  NULL: g computed
                             from W every call (Sec. 3.2.1, per-forward re-quantization).
                             Non-NULL: holds the tied-group g (read only).                 */
    float* a_amax;        /* NVFP4 activation: device FP32 scalar holding the running
                             amax (read only).  Required when afmt == QF_FMT_NVFP4.       */
    uint32_t flags;       /* QF_FLAG_*                                                     */
} qf_qlinear_desc;

/* Bytes of device workspace qf_qlinear_fwd / qf_qlinear_bwd_ste need for `d` (host only). */
QF_API qf_status qf_workspace_size(const qf_qlinear_desc* d, size_t* bytes);

/*
 * qf_saved_size -- bytes of the `saved` buffer of qf_qlinear_fwd / qf_qlinear_bwd_ste (host
 * only): the packed quantized weight and, when afmt != NONE, the packed activation -- the
 * transient quantized operands of Sec. 3.2.1, kept between the forward and the backward in
 * their deployment form (0.5625 bytes per element for NVFP4 / Q4_K, 0.53125 for MXFP4).
 * Layout, each region 256-byte aligned, W's then X's: NVFP4 = {256 B holding the FP32 tensor
 * decode scale S = g / 2688, codes [R, K/2], E4M3 scales [R, K/16]}; MXFP4 = {codes [R, K/2],
 * E8M0 scales [R, K/32]}; Q4_K = {blocks [R, K/256, 144]}; codes and scales as the quantizers
 * write them.
 */
QF_API qf_status qf_saved_size(const qf_qlinear_desc* d, size_t* bytes);

/*
 * qf_qlinear_fwd -- Y = A_hat W_hat^T (Eq. fakequant; bf16 output rounded to nearest even from
 * FP32 accumulation on MFMA; NaN sums give quiet NaNs).
 *   X bf16 [M, K], W bf16 [N, K], Y bf16 [M, N]; ws >= qf_workspace_size bytes, 256-aligned.
 *   saved  device buffer of qf_saved_size(d) bytes, 256-byte aligned, or NULL: receives the
 *          packed W_hat (and A_hat) for the backward; NULL keeps the packed W_hat in the
 *          workspace instead.
 * W is quantized once into its packed codes and scales (Q(W), kept in `saved` or the
 * workspace) and its bf16 W_hat = Q^-1(Q(W)) (the workspace), and Y = A_hat W_hat^T on the bf16
 * MFMA GEMM.  With QF_FLAG_DECODE_IN_GEMM the GEMM instead decodes W_hat from the packed codes
 * in its prologue, stage by stage, into the LDS tiles it multiplies (bit for bit the same
 * x_hat), and no bf16 W_hat goes to memory.  A_hat (afmt != NONE) is quantized to bf16 in the
 * workspace (and to its packed form in `saved`).
 */
QF_API qf_status qf_qlinear_fwd(const qf_qlinear_desc* d, const uint16_t* X, const uint16_t* W,
                                uint16_t* Y, void* saved, void* ws, size_t ws_bytes,
                                qf_stream_t stream);

/*
 * qf_qlinear_fwd_noalloc -- qf_qlinear_fwd without a workspace argument, for callers that
 * cannot allocate device memory (code under HIP graph capture, tight serving loops, harnesses
 * that forbid allocation).  Same kernels and bit-identical Y.  The quantized operands (W_hat,
 * A_hat) and the amax scalar live in a static device array of QF_NOALLOC_SCRATCH_BYTES that
 * the library holds on every device it runs on until the process ends; the call allocates and
 * frees nothing.  Limit: 256 + 2 N K (when wfmt != NONE) + 2 M K (when afmt != NONE) bytes,
 * each operand rounded up to 256, at most QF_NOALLOC_SCRATCH_BYTES (QF_ESHAPE beyond it).
 * Every call on one device shares that device's array and leaves its contents behind: calls
 * that overlap on one device (different streams, or threads) race and must be serialized by
 * the caller.  No QF_FLAG_REUSE_WS backward can follow this call (there is no workspace).
 */
#define QF_NOALLOC_SCRATCH_BYTES (64u << 20)
QF_API qf_status qf_qlinear_fwd_noalloc(const qf_qlinear_desc* d, const uint16_t* X,
                                        const uint16_t* W, uint16_t* Y, qf_stream_t stream);

/*
 * qf_qlinear_bwd_ste -- straight-through backward.
 *   dX = dY W_hat      bf16 [M, K]  (Eq. activation-ste)        dX may be NULL
 *   dW = dY^T A_hat    FP32 [N, K]  (Eq. ste; A_hat = X when afmt == NONE)  dW may be NULL
 * dY is bf16 [M, N] and is not quantized.  dW is overwritten (not accumulated).
 *   saved  the forward's saved buffer (same d, X, W), or NULL: W_hat and A_hat are then
 *          dequantized from their packed form straight into the transposed GEMM operands
 *          (no amax pass, no re-quantization); NULL re-quantizes W and X (or, with
 *          QF_FLAG_REUSE_WS, reuses the workspace).  The gradients are bit-identical either way.
 */
QF_API qf_status qf_qlinear_bwd_ste(const qf_qlinear_desc* d, const uint16_t* dY, const uint16_t* X,
                                    const uint16_t* W, const void* saved, uint16_t* dX, float* dW,
                                    void* ws, size_t ws_bytes, qf_stream_t stream);

/* ---------------------------------------------------------------------------------------
 * Grouped (mixture-of-experts) variant (Sec. 3.3 "Mixture-of-experts adaptation")
 * ------------------------------------------------------------------------------------ */
typedef struct {
    int64_t E;            /* experts                                                       */
    int64_t T;            /* rows of X / Y: tokens x top-k, sorted by expert               */
    int64_t N, K;         /* per-expert weight [N, K]                                      */
    int32_t wfmt, afmt;   /* afmt must be QF_FMT_NONE or QF_FMT_MXFP4                       */
    float* w_amax;        /* NVFP4: device FP32 [E] or NULL (NULL: per-expert g computed)  */
    uint32_t flags;
} qf_grouped_desc;

QF_API qf_status qf_grouped_workspace_size(const qf_grouped_desc* d, size_t* bytes);

/*
 * qf_grouped_saved_size -- bytes of the grouped layer's saved operand (Sec. 3.2.1, Sec. 3.3):
 * the experts' packed W_hat back to back, 0.5625 bytes per element for NVFP4.  Layout, each
 * region 256-byte aligned: NVFP4 = {S [E] (the experts' tensor decode scales), codes [E N, K/2],
 * E4M3 scales [E N, K/16]}; MXFP4 = {codes [E N, K/2], E8M0 scales [E N, K/32]}; Q4_K = {blocks
 * [E N, K/256, 144]}; 0 for an unquantized weight.  Expert e's rows are rows e N .. e N + N - 1.
 * The activations are not saved: the backward forms A_hat's transposed, expert-padded operand
 * from X in one pass, which reads no more than a dequantization of packed codes would.
 */
QF_API qf_status qf_grouped_saved_size(const qf_grouped_desc* d, size_t* bytes);

/*
 * qf_qlinear_grouped_fwd -- for every expert e, rows [off[e], off[e+1]) of X:
 *   Y_e = A_hat_e W_hat_e^T with W_hat_e = Q^-1(Q(W[e])), one tensor scale per expert.
 *   group_offsets: DEVICE int64 [E+1], non-decreasing, off[0] = 0, off[E] = T (the host never
 *   reads it).  X bf16 [T, K], W bf16 [E, N, K], Y bf16 [T, N].
 *   saved: NULL, or a 256-byte aligned device buffer of qf_grouped_saved_size bytes that
 *   receives the experts' packed W_hat (written by the same quantizer launch as W_hat).
 */
QF_API qf_status qf_qlinear_grouped_fwd(const qf_grouped_desc* d, const int64_t* group_offsets,
                                 const uint16_t* X, const uint16_t* W, uint16_t* Y, void* saved,
                                 void* ws, size_t ws_bytes, qf_stream_t stream);

/*
 * qf_qlinear_grouped_bwd_ste -- per expert: dX_e = dY_e W_hat_e (bf16 [T, K], may be NULL),
 *   dW_e = dY_e^T A_hat_e (FP32 [E, N, K], may be NULL; experts with no rows get zeros).
 *   saved: the forward's saved buffer (the experts' W_hat^T are dequantized from it: no amax
 *   pass, no re-quantization), or NULL (W is quantized again, or with QF_FLAG_REUSE_WS the
 *   workspace's W_hat is used).  The gradients are bit-identical either way.
 */
QF_API qf_status qf_qlinear_grouped_bwd_ste(const qf_grouped_desc* d, const int64_t* group_offsets,
                                     const uint16_t* dY, const uint16_t* X, const uint16_t* W,
                                     const void* saved, uint16_t* dX, float* dW, void* ws,
                                     size_t ws_bytes, qf_stream_t stream);

/* ---------------------------------------------------------------------------------------
 * Host-only validation (Sec. 3.2.2: the quantizer interface's preconditions).  Each runs the
 * checks the corresponding entry point runs before it launches anything -- shapes, block
 * multiples, formats, alignment, workspace size -- and returns the status and
 * qf_last_error() message that call would return, without touching the device or reading
 * any tensor.  Pointers are only checked for NULL and alignment.
 * ------------------------------------------------------------------------------------ */
/* A quantizer call: fmt QF_FMT_NVFP4 / MXFP4 / Q4K on x [R, K] with row stride ldx. */
QF_API qf_status qf_validate_fakequant(int fmt, const void* x, int64_t R, int64_t K, int64_t ldx);
/* A layer call pair: d with X, W, Y (dY has Y's shape and stride), saved and ws of ws_bytes. */
QF_API qf_status qf_validate_qlinear(const qf_qlinear_desc* d, const void* X, const void* W,
                                     const void* Y, const void* saved, const void* ws,
                                     size_t ws_bytes);
/* A grouped call pair: d with X [T, K], W [E, N, K], Y [T, N], saved and ws of ws_bytes. */
QF_API qf_status qf_validate_grouped(const qf_grouped_desc* d, const void* X, const void* W,
                                     const void* Y, const void* saved, const void* ws,
                                     size_t ws_bytes);

/*
 * qf_fakequant_transposed -- quantize + dequantize with transposed output: out[k][r] =
 * x_hat[r][k], the x_hat of qf_fakequant_nvfp4 / _mxfp4 / _q4k bit for bit (same per-block
 * equations; blocks run along the rows of x).  The backward of the layer uses it to produce
 * W_hat^T and A_hat^T, the NT-form operands of dX and dW, in one pass.
 *   fmt   QF_FMT_NVFP4, QF_FMT_MXFP4 or QF_FMT_Q4K.
 *   x     bf16 [R, K] (row stride ldx); R % 8 == 0; K a multiple of the format block.
 *   amax  NVFP4: device FP32 tensor amax g, read only (required); ignored otherwise.
 *   out   bf16 [K, R] with row stride ldo >= R (ldo % 8 == 0), 16-byte aligned.
 */
QF_API qf_status qf_fakequant_transposed(int fmt, const uint16_t* x, int64_t R, int64_t K,
                                         int64_t ldx, const float* amax, uint16_t* out,
                                         int64_t ldo, qf_stream_t stream);

/* ---------------------------------------------------------------------------------------
 * Plain BF16 GEMMs on the same MFMA kernels (building blocks of the layer calls above)
 * ------------------------------------------------------------------------------------ */
/*
 * qf_transpose_bf16 -- out[c][r] = in[r][c] for a bf16 [R, C] matrix (row strides ldi, ldo);
 * R and C must be multiples of 8.  The backward uses it to put dY and the quantized operands
 * in the k-contiguous form of the NT GEMM.
 */
QF_API qf_status qf_transpose_bf16(const uint16_t* in, int64_t R, int64_t C, int64_t ldi,
                                   uint16_t* out, int64_t ldo, qf_stream_t stream);

/*
 * qf_gemm_bf16 -- C[M, N] = sum_k opA(m, k) * opB(n, k), FP32 accumulation.
 *   a_kmajor = 1: A stored [M, K] (k contiguous, row stride lda); 0: stored [K, M].
 *   b_kmajor = 1: B stored [N, K] (k contiguous, row stride ldb); 0: stored [K, N].
 *   c_f32 = 1: C is FP32, else bf16 (FP32 sums rounded to nearest even; a NaN sum gives a
 *   quiet NaN whose sign and payload bits are unspecified); row stride ldc.
 * Forward = (1, 1); dX = dY W_hat is (1, 0); dW = dY^T A_hat is (0, 0).
 */
QF_API qf_status qf_gemm_bf16(int64_t M, int64_t N, int64_t K, const uint16_t* A, int64_t lda,
                       int a_kmajor, const uint16_t* B, int64_t ldb, int b_kmajor, void* C,
                       int64_t ldc, int c_f32, qf_stream_t stream);

/*
 * qf_gemm_bf16_at -- qf_gemm_bf16 with A [M, K] and B [N, K] k-contiguous and a bf16 C, that
 * also writes A^T: at[k * ldat + m] = A[m, k] for m < M, k < K (other elements of `at` are
 * left alone).  The layer backward's dX = dY W_hat (Eq. activation-ste) uses it to produce
 * dY^T, the left operand of dW = dY^T A_hat (Eq. ste), from the dY tiles the GEMM stages in
 * LDS anyway, instead of a separate transpose pass over dY.  C and `at` are bit-identical to
 * qf_gemm_bf16 and qf_transpose_bf16.
 *   M and K multiples of 8; ldat >= M, a multiple of 4 and below 2^24; at 16-byte aligned
 *   device memory owned by the caller (needed when M and K are nonzero).
 */
QF_API qf_status qf_gemm_bf16_at(int64_t M, int64_t N, int64_t K, const uint16_t* A, int64_t lda,
                                 const uint16_t* B, int64_t ldb, uint16_t* C, int64_t ldc,
                                 uint16_t* at, int64_t ldat, qf_stream_t stream);

/*
 * qf_gemm_packed_b -- C[M, N] = A W_hat^T with W_hat decoded inside the GEMM from the packed
 * weight (the layer forward's product, Eq. fakequant with Q^-1 in the GEMM's prologue): each
 * 64-deep stage of the B tile is decoded from codes and scales by the quantizers' own decode
 * and written to LDS, so C equals qf_gemm_bf16 on the bf16 x_hat of qf_fakequant_* bit for bit.
 *   A      bf16 [M, K], k contiguous, row stride lda.
 *   fmt    QF_FMT_NVFP4 (codes [N, K/2], E4M3 scales [N, K/16], S = the FP32 tensor decode
 *          scale g / 2688 on the device, as qf_fakequant_nvfp4's s_out), QF_FMT_MXFP4 (codes,
 *          E8M0 scales [N, K/32]; S ignored) or QF_FMT_Q4K (blocks [N, K/256, 144] in codes;
 *          scales and S ignored), each dense row-major as the quantizers write them.
 *   C      bf16 [M, N], row stride ldc.
 *   K a multiple of 64 (Q4K: 256); codes / scales 16-byte aligned.
 */
QF_API qf_status qf_gemm_packed_b(int64_t M, int64_t N, int64_t K, const uint16_t* A,
                                  int64_t lda, int fmt, const uint8_t* codes,
                                  const uint8_t* scales, const float* S, uint16_t* C,
                                  int64_t ldc, qf_stream_t stream);

/*
 * qf_dequantize_transposed -- out[k][r] = x_hat[r][k] decoded from a packed [R, K] tensor
 * (Eqs. nvfp4-dequant, mxfp4-dequant, q4k-dequant; the layer backward's transposed operands
 * from the saved buffer): bit for bit qf_fakequant_transposed of the tensor the codes came
 * from.  fmt, codes, scales, S as for qf_gemm_packed_b; R % 8 == 0; out bf16 [K, R] with row
 * stride ldo >= R (ldo % 8 == 0), 16-byte aligned.
 */
QF_API qf_status qf_dequantize_transposed(int fmt, const uint8_t* codes, const uint8_t* scales,
                                          const float* S, int64_t R, int64_t K, uint16_t* out,
                                          int64_t ldo, qf_stream_t stream);

/*
 * Fragment-major B operand: B [N, K] stored as the v_mfma_f32_32x32x16_bf16 operands of 32-row
 * by 16-column blocks, blocks ordered row-block-major: element (n, k) at
 *   ((n / 32) (K / 16) + k / 16) * 512 + ((n % 32) + 32 ((k / 8) % 2)) * 8 + k % 8,
 * rows past N (up to the next multiple of 32) zero.  A GEMM reading B in this form loads each
 * wavefront's operand of one 16-deep slice as one contiguous 1 KB block straight into the
 * matrix cores' registers and stages only A in LDS (half of the LDS traffic of the k-contiguous
 * form).  K % 16 == 0 for the layout, K % 64 == 0 for the GEMM.
 * qf_fragment_bytes: bytes of the layout (host only).
 * qf_pack_fragments: out (fragment-major) from B [N, K] row-major with row stride ldb
 *   (16-byte aligned, ldb % 8 == 0).
 * qf_gemm_bf16_fragb: C[M, N] = A B^T with A [M, K] k-contiguous (row stride lda) and B in the
 *   fragment-major layout; bf16 or FP32 C as qf_gemm_bf16_ws (same split of a partial last round
 *   with the workspace); bit-identical to qf_gemm_bf16 on the row-major B.
 */
QF_API qf_status qf_fragment_bytes(int64_t N, int64_t K, size_t* bytes);
QF_API qf_status qf_pack_fragments(const uint16_t* B, int64_t N, int64_t K, int64_t ldb,
                                   uint16_t* out, qf_stream_t stream);
QF_API qf_status qf_gemm_bf16_fragb(int64_t M, int64_t N, int64_t K, const uint16_t* A,
                                    int64_t lda, const uint16_t* Bf, void* C, int64_t ldc,
                                    int c_f32, void* ws, size_t ws_bytes, qf_stream_t stream);

/*
 * qf_gemm_workspace_size / qf_gemm_bf16_ws -- qf_gemm_bf16 with a caller workspace.  With
 * k-contiguous A and B and an FP32 C (the dW product), a last round of output tiles that
 * would leave at least half of the compute units idle is computed as two K-halves into the
 * workspace and summed in a fixed order (deterministic; the summation order differs from the
 * unsplit call by that one split).  Other layouts ignore the workspace.  ws: device memory,
 * 256-byte aligned, at least the returned size (0 when no split can happen); ownership stays
 * with the caller.
 */
QF_API qf_status qf_gemm_workspace_size(int64_t M, int64_t N, int c_f32, size_t* bytes);
QF_API qf_status qf_gemm_bf16_ws(int64_t M, int64_t N, int64_t K, const uint16_t* A, int64_t lda,
                                 int a_kmajor, const uint16_t* B, int64_t ldb, int b_kmajor,
                                 void* C, int64_t ldc, int c_f32, void* ws, size_t ws_bytes,
                                 qf_stream_t stream);

/* ---------------------------------------------------------------------------------------
 * LoRA-QAD (Sec. 3.3 "Full-parameter vs. LoRA-QAD", Eqs. qad-lora and export-lora;
 * "Mixture-of-experts adaptation")
 * ------------------------------------------------------------------------------------ */
/*
 * Low-rank adapters of a frozen bf16 weight W [N, K]: the student's weight is the merged
 * W + scale * B A, quantized as a whole (W_hat = Q^-1(Q(W + scale B A)), Eq. qad-lora); the
 * exporter quantizes the same merged weight (Eq. export-lora).
 *   A      FP32 [r, K] (row stride K), device, 16-byte aligned.
 *   B      FP32 [N, r] (row stride r), device, 16-byte aligned.
 *   r      rank, 1 <= r <= 4096.
 *   scale  multiplies B A (1 for the paper's W + B A; LoRA's alpha / r otherwise).
 *   a_shared, b_shared  grouped (MoE) calls only: 0 = one factor per expert (A [E, r, K],
 *          B [E, N, r]), 1 = one factor shared by every expert (A [r, K] / B [N, r]); the
 *          paper's hybrid layout shares A for gate/up and B for down.  Ignored elsewhere.
 * Merge arithmetic (exactly what the library computes): per element, acc = sum over
 * j = 0..r-1 of B[n][j] A[j][k] in binary32 with one fused multiply-add per term in rising
 * j, then bf16(W[n][k] + fl(scale * acc)) rounded to nearest even.  The merged weight is
 * never written to memory by the layer calls.
 */
typedef struct {
    const float* A;
    const float* B;
    int64_t r;
    float scale;
    int32_t a_shared, b_shared;
} qf_lora;

/*
 * qf_lora_amax -- g = max |W + scale B A| over the merged bf16 weight (the NVFP4 tensor
 * amax of Eq. qad-lora); accumulate as in qf_amax (tied groups: call once per member).
 */
QF_API qf_status qf_lora_amax(const uint16_t* W, int64_t N, int64_t K, int64_t ldw,
                              const qf_lora* lora, float* amax, int accumulate,
                              qf_stream_t stream);

/*
 * qf_lora_fakequant -- quantize + dequantize the merged weight W + scale B A (Eqs. qad-lora,
 * export-lora) with the per-block equations of qf_fakequant_nvfp4 / _mxfp4 / _q4k.
 *   fmt     QF_FMT_NONE (xhat = the merged bf16 weight), NVFP4, MXFP4 or Q4K.
 *   amax, amax_mode, s_out   NVFP4 only, as in qf_fakequant_nvfp4 (COMPUTE: g of the merged
 *           weight); ignored (may be NULL) for the other formats.
 *   codes [N, K/2], scales [N, K/16 | K/32]   NVFP4 / MXFP4 export outputs, or NULL.
 *   packed [N, K/256, 144]   Q4_K export blocks, or NULL.
 *   xhat  bf16 [N, K] (row stride K), or NULL.
 * An output that the format does not produce must be NULL (QF_EINVAL otherwise).
 */
QF_API qf_status qf_lora_fakequant(int fmt, const uint16_t* W, int64_t N, int64_t K,
                                   int64_t ldw, const qf_lora* lora, float* amax, int amax_mode,
                                   float* s_out, uint8_t* codes, uint8_t* scales,
                                   uint8_t* packed, uint16_t* xhat, qf_stream_t stream);

/*
 * qf_lora_fakequant_transposed -- out[k][n] = x_hat[n][k] of qf_lora_fakequant, bit for bit
 * (the dX operand of the backward in NT form).  fmt NVFP4 / MXFP4 / Q4K (or NONE: the
 * merged weight transposed); amax: NVFP4 tensor amax (read only, required for NVFP4).
 * N % 8 == 0; out bf16 [K, N] with row stride ldo >= N (ldo % 8 == 0).
 */
QF_API qf_status qf_lora_fakequant_transposed(int fmt, const uint16_t* W, int64_t N, int64_t K,
                                              int64_t ldw, const qf_lora* lora,
                                              const float* amax, uint16_t* out, int64_t ldo,
                                              qf_stream_t stream);

/* Workspace bytes of qf_qlinear_lora_fwd / _bwd_ste for (d, lora) (host only). */
QF_API qf_status qf_lora_workspace_size(const qf_qlinear_desc* d, const qf_lora* lora,
                                        size_t* bytes);

/*
 * qf_qlinear_lora_fwd -- Y = A_hat W_hat^T with W_hat = Q^-1(Q(W + scale B A)) (Eq. qad-lora;
 * A_hat as in qf_qlinear_fwd).  d as for qf_qlinear_fwd (wfmt may be NONE: bf16 LoRA);
 * NVFP4 with d->w_amax == NULL uses g of the merged weight.  W is the frozen base weight.
 * The workspace keeps W_hat and A_hat for a backward with QF_FLAG_REUSE_WS.
 */
QF_API qf_status qf_qlinear_lora_fwd(const qf_qlinear_desc* d, const qf_lora* lora,
                                     const uint16_t* X, const uint16_t* W, uint16_t* Y, void* ws,
                                     size_t ws_bytes, qf_stream_t stream);

/*
 * qf_qlinear_lora_bwd_ste -- straight-through backward of the LoRA layer.  The merged weight's
 * STE gradient is G = dY^T A_hat (Eq. ste); the frozen W gets none, the factors get
 *   dB = scale G A^T    FP32 [N, r]       dA = scale B^T G    FP32 [r, K]
 * (overwritten; either may be NULL), and dX = dY W_hat (Eq. activation-ste; bf16 [M, K], may
 * be NULL).  G itself is never formed: dB = scale dY^T (A_hat A^T), dA = scale (dY B)^T A_hat.
 * The rank-r products accumulate in FP32 on the matrix cores, each FP32 factor (and rank-r
 * intermediate) taken as the sum of two bf16 halves (relative error below 2^-17 per value), in
 * a fixed order, so the gradients are deterministic.
 */
QF_API qf_status qf_qlinear_lora_bwd_ste(const qf_qlinear_desc* d, const qf_lora* lora,
                                         const uint16_t* dY, const uint16_t* X,
                                         const uint16_t* W, uint16_t* dX, float* dA, float* dB,
                                         void* ws, size_t ws_bytes, qf_stream_t stream);

/*
 * Grouped LoRA-QAD (Sec. 3.3 "Mixture-of-experts adaptation"): expert e's weight is the merged
 * W[e] + scale B_e A_e, quantized per expert (its own NVFP4 tensor amax unless d->w_amax holds
 * tied values [E]).  lora->a_shared / b_shared select one factor for all experts (A [r, K] /
 * B [N, r]) instead of one per expert (A [E, r, K] / B [E, N, r]); the paper's hybrid layout
 * shares A for gate/up and B for down.  group_offsets, X, W, Y, d as for the grouped layer
 * (afmt NONE or MXFP4).  The merged weights are never written to memory.
 * Backward: dX = dY_e W_hat_e per expert (bf16 [T, K], may be NULL); dA, dB FP32 shaped like
 * A, B (overwritten; may be NULL): an unshared factor gets its expert's gradient
 * (dB_e = scale dY_e^T A_hat_e A_e^T, dA_e = scale B_e^T dY_e^T A_hat_e; zeros for an expert
 * with no rows), a shared factor the sum over experts.
 */
QF_API qf_status qf_grouped_lora_workspace_size(const qf_grouped_desc* d, const qf_lora* lora,
                                                size_t* bytes);
QF_API qf_status qf_qlinear_grouped_lora_fwd(const qf_grouped_desc* d, const qf_lora* lora,
                                             const int64_t* group_offsets, const uint16_t* X,
                                             const uint16_t* W, uint16_t* Y, void* ws,
                                             size_t ws_bytes, qf_stream_t stream);
QF_API qf_status qf_qlinear_grouped_lora_bwd_ste(const qf_grouped_desc* d, const qf_lora* lora,
                                                 const int64_t* group_offsets,
                                                 const uint16_t* dY, const uint16_t* X,
                                                 const uint16_t* W, uint16_t* dX, float* dA,
                                                 float* dB, void* ws, size_t ws_bytes,
                                                 qf_stream_t stream);

/* ---------------------------------------------------------------------------------------
 * QAD distillation loss (Sec. 3.3 "Quantization-aware distillation", Eq. qad-objective)
 * ------------------------------------------------------------------------------------ */
/*
 * qf_qad_kl -- token-averaged forward KL between the teacher's and the student's softmax
 * distributions over the vocabulary, its gradient with respect to the student's logits, and
 * the teacher-student top-1 agreement (a training metric of Sec. 4).
 *   zt, zs     bf16 logits [L, V] of the frozen teacher and of the student (row strides ldt,
 *              lds, multiples of 8); V % 8 == 0; logits must be finite.
 *   row_kl     FP32 [L], required: KL_t = sum_v p_T log(p_T / p_S) per token (FP32 online
 *              log-sum-exp statistics; deterministic order).
 *   loss       FP32 device scalar or NULL: (1/L) sum_t KL_t.
 *   grad       bf16 [L, V] (row stride ldg) or NULL: grad_scale * (p_S - p_T); with
 *              grad_scale = 1/L this is d loss / d z_S.
 *   agree      int32 [L] or NULL: 1 where the first maximum of z_T and of z_S are at the
 *              same index, else 0.
 * L = 0 gives loss 0.
 */
QF_API qf_status qf_qad_kl(const uint16_t* zt, int64_t ldt, const uint16_t* zs, int64_t lds,
                           int64_t L, int64_t V, float grad_scale, float* row_kl, float* loss,
                           uint16_t* grad, int64_t ldg, int32_t* agree, qf_stream_t stream);

/* ---------------------------------------------------------------------------------------
 * Engine-native export and weight sync (Sec. 3.5; Sec. 3.2.3 "Engine-specific scale sharing";
 * Sec. 3.4 "Low-precision weight synchronization")
 * ------------------------------------------------------------------------------------ */
typedef struct {
    const uint16_t* W;    /* bf16 [rows, K], row stride ldw (device) */
    int64_t rows;
    int64_t ldw;
} qf_member;

/*
 * qf_export_fused -- export of a fused projection (attention QKV, MLP gate/up): the engine's
 * fused weight is the row concatenation of the n member weights (1 <= n <= 8, common K).
 *   fmt        QF_FMT_NVFP4 or QF_FMT_MXFP4.
 *   codes      [N, K/2] (N = sum of rows; element 2i in the low nibble), required.
 *   scales     [N, K/16] E4M3 (NVFP4) or [N, K/32] E8M0 (MXFP4), required.
 *   NVFP4 only:
 *   w_amax     device FP32 scalar, required: receives the tied amax g over all members.
 *   weight_scale_2  device FP32 scalar or NULL: the tied tensor decode scale g / 2688 (one
 *              for the fused matrix, as the engine uses it).
 *   a_amax, input_scale  device FP32 scalars or NULL: input_scale = a_amax / 2688, the
 *              static activation scale exported from the running activation amax (NVFP4
 *              paragraph) -- the decode scale the activation quantizer uses for that amax.
 * The codes and block scales equal those of qf_fakequant_nvfp4 / _mxfp4 on the concatenated
 * weight, bit for bit.  Any output may point into a weight-sync payload (below).
 */
QF_API qf_status qf_export_fused(int fmt, const qf_member* members, int n, int64_t K,
                                 uint8_t* codes, uint8_t* scales, float* w_amax,
                                 float* weight_scale_2, const float* a_amax, float* input_scale,
                                 qf_stream_t stream);

/*
 * Weight-sync payload of one layer (this library's format; the transport is the caller's):
 * one contiguous byte buffer with a 64-byte header, then the codes, the block scales and two
 * FP32 scalars {weight_scale_2, input_scale} (zeros for MXFP4), each section at a multiple of
 * 256 bytes.  Header (little-endian): u32 magic 0x31504651 ("QFP1"), u32 format, i64 N,
 * i64 K, u64 offsets of codes, scales and scalars, u64 total bytes, 8 bytes zero.
 * qf_payload_layout_of (host only) returns the offsets and size; qf_export_fused (or the
 * quantizers) write the sections in place; qf_payload_write_header writes the header and
 * leaves the sections untouched.
 */
typedef struct {
    uint64_t codes, scales, scalars, total;
} qf_payload_layout;
QF_API qf_status qf_payload_layout_of(int fmt, int64_t N, int64_t K, qf_payload_layout* out);
QF_API qf_status qf_payload_write_header(int fmt, int64_t N, int64_t K, void* payload,
                                         qf_stream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* QF_H */
