/*
 * qlinear.h — block-quantized linear layers (int8 / 4-bit weights with
 * per-block fp16 scales) for AMD Instinct MI355X (gfx950).
 *
 * The operation (paper: Methodology, "The aria runtime" and "Quantization
 * and its evaluation"): the diffusion transformer's weights are stored as
 * 8-bit or 4-bit integers (q8 / q4) instead of half precision; the
 * compressed copy owns its own memory so that the full-precision source can
 * be released once packed, and the linear layers are evaluated from it.  The
 * paper does not fix the encoding; this library uses symmetric absmax
 * quantization over blocks of 32 consecutive weights along the reduction
 * dimension K with one fp16 scale per block:
 *
 *     s[n][b] = fp16 nearest to max_{k in b} |W[n][k]| / Q   (ties to even)
 *     c[n][k] = clamp(nearest integer to W[n][k] / s[n][b], -Q, Q)
 *               (ties to even; all codes 0 when s == 0)
 *     Q = 127 (QL_FMT_INT8) or 7 (QL_FMT_Q4)
 *
 * and the forward product of one linear layer (no bias)
 *
 *     Y[m][n] = sum_b s[n][b] * sum_{k in b} X[m][k] * c[n][k]
 *
 * with W [N][K] (out x in, like a framework's Linear weight), X [M][K] and
 * Y [M][N], all row-major.
 *
 * Accuracy of the forward product against the exact sum above: fp32
 * activations, and bf16 activations at M <= 256 (or when K % 256 != 0 or
 * an operand is not 16-byte aligned), are contracted with the exact codes
 * and fp32 block partials (error a few fp32 roundings).  bf16 activations
 * at larger M take the fp16 path: X is copied
 * exactly to fp16 with a power-of-two shift per row, each weight enters the
 * matrix cores as fp16(c * fp16(s * 2^f)) with one shift f per weight row
 * and K part (the library may cut a long reduction into parts; Q * max_b s
 * * 2^f in [2^14, 2^15) over the row's blocks in the part), so the one extra
 * rounding is that of c * s to 11 significant bits: relative error at most
 * 2^-11 per weight for every block whose scale is at least Q * 2^-28 of the
 * largest scale of its row in its part, a fortiori of its row (2^-21 for
 * int8, 2^-25 for q4).  Smaller blocks' scaled scales are fp16 subnormals;
 * their weights are off by less than 2^-31 of the row's largest dequantized
 * weight.  Measured: about 2e-4 of max |Y| at transformer shapes.
 *
 * Data formats (all buffers are DEVICE memory owned by the caller):
 *   W       fp32 [N][K]
 *   codes   QL_FMT_INT8: int8 [N][K], two's complement
 *           QL_FMT_Q4:   uint8 [N][K/2]; byte j of a row holds code 2j in its
 *                        low nibble and code 2j+1 in its high nibble, both
 *                        two's complement (the stored codes -128 / -8 are
 *                        accepted by the forward pass, never produced)
 *           QL_FMT_F16:  fp16 bit patterns, uint16 [N][K] -- unquantized
 *                        weights, the reference point the paper's table of
 *                        precisions measures q8 / q4 against (Experiments,
 *                        runtime benchmarks); forward only, bf16
 *                        activations, K % 256 == 0 (else
 *                        QL_ERR_UNSUPPORTED), scales unused (may be NULL);
 *                        Y = X * W^T on the fp16 path (X shifted to fp16
 *                        exactly, the weights exact, fp32 accumulation)
 *   scales  fp16 bit patterns, uint16 [N][K/32]
 *   X       QL_DT_BF16: bf16 bit patterns, uint16 [M][K]; QL_DT_F32: fp32
 *   Y       fp32 [M][N]
 *
 * Conventions shared by every entry point:
 *   - Every function returns a ql_status (an int) and never aborts or throws.
 *   - All argument checks happen before anything is enqueued; a call that
 *     returns an error has enqueued nothing.
 *   - Alignment: codes and X must be 16-byte aligned, scales 2-byte and Y
 *     4-byte aligned (2-byte for bf16 Y); the entry points after
 *     qlinear_block_forward state their own rules (QL_ERR_ALIGN otherwise).
 *   - Work runs on the caller's HIP stream; only qlinear_quantize waits for
 *     its own work.  Buffers must stay alive until the stream has passed the
 *     enqueued work.  Asynchronous device faults surface at the caller's next
 *     synchronization, as in HIP itself.
 *   - The library keeps no pointer to caller memory after a call returns.
 *   - Workspace: the fp16 path (above) needs M * K * 2 + M * 4 bytes per
 *     distinct activation tensor of a call, plus fp32 partial results when
 *     it splits a layer's reduction.  The library keeps one workspace per
 *     (device, stream), taken from a stream-ordered memory pool it owns; it
 *     grows when a call outside graph capture needs more (the old buffer
 *     goes back to the pool in stream order), so steady-state calls
 *     allocate nothing.  Consequences: calls on one stream share it, which
 *     their stream order makes safe; a graph captured on a stream keeps
 *     that stream's buffer (it is then never released before the process
 *     ends), so replays of the graph must not overlap calls on the capture
 *     stream or replays of other graphs captured on it.  A call under
 *     capture that needs more than its stream's buffer allocates for itself
 *     from the pool (allocation and free nodes in the graph) instead.  A
 *     destroyed stream's handle value, if reused, inherits its buffer.  No
 *     other forward path uses device memory beyond its arguments.
 *     Allocation failure returns QL_ERR_HIP.
 */
#ifndef QLINEAR_H
#define QLINEAR_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    QL_OK = 0,
    QL_ERR_INVALID = 1,     /* null pointer, unknown enum value, n_lin out of range */
    QL_ERR_SHAPE = 2,       /* K % 32 != 0, N <= 0, K <= 0, M < 0 */
    QL_ERR_ALIGN = 3,       /* pointer alignment (see above) */
    QL_ERR_RANGE = 4,       /* weight NaN/Inf, or a block's scale overflows fp16 */
    QL_ERR_UNSUPPORTED = 5, /* size beyond what the kernels index (see below) */
    QL_ERR_HIP = 6          /* a HIP runtime call or kernel launch failed */
} ql_status;

typedef enum { QL_FMT_Q4 = 4, QL_FMT_INT8 = 8, QL_FMT_F16 = 16 } ql_fmt;
                                               /* q4 / int8: block fixed at 32 along K */
typedef enum { QL_DT_F32 = 0, QL_DT_BF16 = 1 } ql_dtype; /* activation dtype; Y is fp32 */

#define QL_BLOCK 32

/* Bytes of the packed codes of an N x K weight: N*K (int8), N*K/2 (q4) or
 * 2*N*K (the fp16 weights of QL_FMT_F16).  Returns 0 for an unknown format
 * or a non-positive size. */
size_t qlinear_codes_bytes(int fmt, int64_t N, int64_t K);

/* Bytes of the fp16 scales of an N x K weight: N * (K/32) * 2.
 * Returns 0 when K % 32 != 0 or a size is non-positive. */
size_t qlinear_scales_bytes(int64_t N, int64_t K);

/* Quantize W (fp32 [N][K], device) into codes and scales (device), by the
 * rule at the top of this file.  Synchronous: waits for its own work on
 * `stream` and reports QL_ERR_RANGE if W holds a NaN/Inf or a block's
 * scale rounds to +inf (absmax / Q >= 65520); the outputs are then
 * unspecified.  Once it returns QL_OK the caller may free W: the codes and
 * scales replace the full-precision copy (paper: the compressed copy owns its
 * memory and the source is released once packed).  Allocates and frees one
 * 4-byte device status word per call (a load-time operation, not a per-step
 * one).  Sizes: N * K < 2^40. */
int qlinear_quantize(int fmt, const float *W, int64_t N, int64_t K,
                     void *codes, uint16_t *scales, hipStream_t stream);

/* Y[M][N] (fp32) = X[M][K] * dequant(codes, scales)^T, the forward pass of
 * one quantized linear layer.  Asynchronous on `stream`; does not
 * synchronize, and allocates nothing outside the workspace described
 * above.  M == 0 is a successful no-op.  Y must not alias
 * X, codes or scales.  Sizes: M, N < 2^31, K < 2^31. */
int qlinear_forward(int fmt, const void *X, int xdt, int64_t M, int64_t K,
                    const void *codes, const uint16_t *scales, int64_t N,
                    float *Y, hipStream_t stream);

/* One quantized linear layer for qlinear_block_forward. */
typedef struct {
    int fmt;                /* ql_fmt */
    const void *X;          /* [M][K], dtype xdt */
    int xdt;                /* ql_dtype */
    int64_t M, K, N;
    const void *codes;
    const uint16_t *scales;
    float *Y;               /* [M][N] */
} ql_linear;

#define QL_MAX_GROUP 8

/* The linear layers of one transformer block (QKV projection, attention
 * output, FFN up and FFN down: the set the paper quantizes) evaluated as one
 * grouped launch.  The n_lin (1..QL_MAX_GROUP) products are independent:
 * no Y may alias any X, codes, scales or other Y of the group.  Layers that
 * share fmt and xdt run in one launch over their combined tiles; otherwise
 * the call falls back to one launch per layer; layers reading the same X
 * share its fp16 copy.  Asynchronous on `stream`, workspace as above.  Each
 * entry is checked as in qlinear_forward. */
int qlinear_block_forward(const ql_linear *lin, int n_lin, hipStream_t stream);

/* Epilogue of a linear layer: the rest of the DiT block's linear around the
 * product (bias, the feed-forward's GELU, the residual adds of the stream
 * the paper steers: Methodology, taste steering), applied by the kernel
 * that stores each output element:
 *
 *     Y[m][n] = act(P[m][n] + bias[n]) + residual[m][n]
 *               (+ alpha * steer_norm * steer_dir[n], see below)
 *
 * with P the product of qlinear_forward, in fp32.  act: QL_ACT_NONE, or
 * QL_ACT_GELU in its exact form x * (1 + erf(x / sqrt 2)) / 2.  bias fp32
 * [N] and residual fp32 [M][N] may each be NULL (4-byte aligned).  ydt:
 * QL_DT_F32 (Y fp32 [M][N]) or QL_DT_BF16 (Y bf16 bit patterns [M][N],
 * rounded to nearest even from the fp32 result; 2-byte aligned Y).
 * residual may be Y itself when ydt is QL_DT_F32 (an in-place residual
 * add); no other aliasing. */
typedef enum { QL_ACT_NONE = 0, QL_ACT_GELU = 1 } ql_act;

typedef struct {
    const float *bias;      /* [N] or NULL */
    int act;                /* ql_act */
    const float *residual;  /* [M][N] or NULL */
    int ydt;                /* ql_dtype of Y */
    /* Steering (Methodology, additive injection, Eq. 2) on the block's
     * output: + alpha * steer_norm * steer_dir[n], alpha = *steer_strength
     * read from device memory by every launch (a captured graph picks up a
     * new strength without re-capture); skipped, bit for bit, when alpha is
     * 0.  steer_dir: unit direction fp32 [N] (4-byte aligned) or NULL for
     * none; steer_norm: the layer's mean residual norm ||h_bar||. */
    const float *steer_dir;
    float steer_norm;
    const float *steer_strength;  /* device fp32 scalar; required with steer_dir */
    /* Optional bf16 copy of the output (fp32 Y only): y_bf16_copy[m][n] =
     * Y[m][n] rounded to nearest even, bf16 bit patterns [M][N], 2-byte
     * aligned (8-byte for the vector store paths), aliasing no other
     * argument; NULL for none.  With Y the residual stream this is the next
     * linear layer's bf16 input, written by the same kernel. */
    uint16_t *y_bf16_copy;
} ql_epilogue;

/* qlinear_forward with an epilogue (ep == NULL: none, fp32 Y).  Y is fp32 or
 * bf16 as ep->ydt says.  Errors as in qlinear_forward, plus QL_ERR_INVALID
 * for an unknown act or ydt and QL_ERR_ALIGN for misaligned bias/residual. */
int qlinear_forward_ep(int fmt, const void *X, int xdt, int64_t M, int64_t K,
                       const void *codes, const uint16_t *scales, int64_t N,
                       void *Y, const ql_epilogue *ep, hipStream_t stream);

/* One layer of qlinear_block_forward_ep: lin.Y points to fp32 or bf16
 * outputs as ep.ydt says. */
typedef struct {
    ql_linear lin;
    ql_epilogue ep;
} ql_linear_ep;

/* qlinear_block_forward with an epilogue per layer. */
int qlinear_block_forward_ep(const ql_linear_ep *lin, int n_lin, hipStream_t stream);

/* qlinear_block_forward_ep for callers that cannot allocate device memory
 * (code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc).  The same kernels and results, bit for bit, but the
 * workspace (fp16 activation copies, row shifts, split partials and arrival
 * counters) lives in a static device array of the library, 128 MiB
 * (134217728 bytes) per device, held from the first call on a device until
 * the process ends.  The call allocates and frees nothing, through HIP or
 * any allocating library.  A call whose workspace would exceed the array
 * returns QL_ERR_UNSUPPORTED and enqueues nothing (at d = 2048 and 2048
 * tokens one block's grouped call takes about 76 MB, the FFN-down layer
 * alone about 101 MB; a block at 4096 tokens about 84 MB).  Every
 * call on a device shares that device's array: calls that may overlap on
 * one device (different streams, or graph replays concurrent with other
 * calls) race and must be ordered by the caller; calls on one stream are
 * ordered by the stream.  The array keeps the last call's contents; the
 * kernels clear what must start at zero themselves.  Other arguments,
 * checks and errors as qlinear_block_forward_ep; QL_ERR_HIP if the array's
 * device address cannot be looked up. */
int qlinear_block_forward_ep_noalloc(const ql_linear_ep *lin, int n_lin, hipStream_t stream);

/* ---- W8A8: int8 activations against int8 weights -------------------------
 *
 * The paper's 8-bit-arithmetic mode (Methodology; Table II): activations are
 * quantized alongside the weights and the products run on the integer
 * matrix cores.  Activation granularity (the paper states none): one scale
 * per token, sx[m] = fp16 nearest to max_k |X[m][k]| / 127 (ties to even),
 * q[m][k] = nearest integer to X[m][k] / sx[m] (ties to even), clamped to
 * [-127, 127]: the weight rules with the whole row as the block.  Weights:
 * QL_FMT_INT8 codes and scales as produced by qlinear_quantize.  Then
 *
 *     Y[m][n] = sx[m] * sum_b s[n][b] * sum_{k in block b} q[m][k] * c[n][k]
 *
 * with each block's integer sum exact and the block sum accumulated in
 * fp32. */

/* Per-token int8 quantization of X [M][K] (fp32 or bf16 bits, 16-byte
 * aligned, K % 32 == 0) into qx int8 [M][K] (16-byte aligned) and sx fp16
 * bits [M] (2-byte aligned).  Asynchronous on `stream`; M == 0 is a no-op.
 * A row holding a NaN or Inf, or whose scale would exceed the fp16 range
 * (max |x| >= 65520 * 127), gets the NaN scale 0x7E00 and zero codes, so
 * that its outputs are NaN: there is no synchronous status. */
int qlinear_quantize_act(const void *X, int xdt, int64_t M, int64_t K, int8_t *qx,
                         uint16_t *sx, hipStream_t stream);

/* Y = the W8A8 product of (qx, sx) [M][K] and int8 weights (codes [N][K],
 * 16-byte aligned; scales [N][K/32]), then the epilogue ep (NULL: none, fp32
 * Y).  Asynchronous; K % 32 == 0; Y must not alias an input (except
 * ep->residual as for qlinear_forward_ep).  Errors as qlinear_forward_ep. */
int qlinear_forward_w8a8(const int8_t *qx, const uint16_t *sx, int64_t M, int64_t K,
                         const void *codes, const uint16_t *scales, int64_t N, void *Y,
                         const ql_epilogue *ep, hipStream_t stream);

/* The steering injection alone (Methodology, additive injection, Eq. 2):
 * h[m][n] += alpha * hnorm * dir[n] on the residual stream h fp32 [M][N] in
 * place, alpha = *strength read from device memory at run time; nothing is
 * written when alpha is 0 (h stays bit for bit).  dir: unit direction fp32
 * [N].  Pointers 4-byte aligned; h must not alias dir or strength.
 * Asynchronous on `stream`; M == 0 is a no-op. */
int qlinear_steer(float *h, int64_t M, int64_t N, const float *dir, float hnorm,
                  const float *strength, hipStream_t stream);

/* ---- self-attention ------------------------------------------------------
 *
 * The DiT block's self-attention (Methodology: the GPU path's attention; a
 * FlashAttention-class fused kernel is the open lever the paper names), in
 * one pass over the keys with a running maximum and sum:
 *
 *     O[b,t,h,:] = sum_j p_j V[b,j,h,:] / sum_j p_j,
 *     p_j = exp(s_j - max_i s_i),  s_j = scale * <Q[b,t,h,:], K[b,j,h,:]>
 *
 * over all T keys of sequence b (no mask), scale >= 0 and finite
 * (QL_ERR_INVALID otherwise).  Q, K, V: bf16 bit patterns;
 * row b * T + t of Q starts at q + (b * T + t) * ldq and head h at column
 * h * dh (likewise K, V), so the fused [tokens][3 d] output of a QKV linear
 * is read in place (q = qkv, k = qkv + d, v = qkv + 2 d, ld = 3 d).  O: rows
 * of ldo elements, fp32 or bf16 (odt).  Head dimension 64 only
 * (QL_ERR_UNSUPPORTED otherwise); B * H <= 65535, B * T < 2^31 and
 * ceil(T / 128) * B * H < 2^31 (likewise).  q, k, v 16-byte aligned
 * with ld % 8 == 0; o 16-byte (fp32) or 8-byte (bf16) aligned with
 * ldo % 4 == 0.  The probabilities enter the value product rounded to bf16
 * (fp32 accumulation).  Asynchronous on `stream`. */
int qlinear_attention(const uint16_t *q, int64_t ldq, const uint16_t *k, int64_t ldk,
                      const uint16_t *v, int64_t ldv, int64_t B, int64_t T, int64_t H,
                      int64_t dh, float scale, void *o, int64_t ldo, int odt,
                      hipStream_t stream);

/* ---- kernel path selection (diagnostics and tests) -----------------------
 *
 * The forward product of the quantized formats has several kernels, each
 * exact to its own stated accuracy over the shapes it takes; the library
 * normally picks one by shape (see the accuracy paragraph at the top).
 * qlinear_force_path makes every later call of qlinear_forward[_ep] and
 * qlinear_block_forward[_ep] on quantized weights use one kernel, so that
 * the kernels can be run on the same inputs and compared:
 *   QL_PATH_GEMV    wavefront-reduction GEMV: bf16 X, 1 <= M <= 4,
 *                   K % 256 == 0, K <= 8192
 *   QL_PATH_STREAM  weight-streaming kernel: bf16 X, M <= 32, K % 256 == 0,
 *                   K <= 2^24, 16-byte aligned scales
 *   QL_PATH_SKINNY  few-row exact MFMA kernel: bf16 X, M <= 64
 *   QL_PATH_TILED   tiled exact MFMA kernel: any M, bf16 or fp32 X
 *   QL_PATH_WIDE    the large-M fp16 path: bf16 X, K % 256 == 0,
 *                   K < 2^23, 16-byte aligned scales
 *   QL_PATH_MID     the mid-M exact kernel (the normal choice for
 *                   32 < M <= 256): bf16 X, K % 256 == 0, K < 2^23,
 *                   16-byte aligned X, codes and scales
 * A call whose layers a forced kernel cannot take returns
 * QL_ERR_UNSUPPORTED and enqueues nothing.  fp16 weights (QL_FMT_F16) are
 * not affected.  The setting is process-wide (not per thread or stream);
 * QL_PATH_AUTO restores the normal choice.  Returns QL_ERR_INVALID for an
 * unknown value. */
typedef enum {
    QL_PATH_AUTO = 0,
    QL_PATH_GEMV = 1,
    QL_PATH_STREAM = 2,
    QL_PATH_SKINNY = 3,
    QL_PATH_TILED = 4,
    QL_PATH_WIDE = 5,
    QL_PATH_MID = 6
} ql_path;

int qlinear_force_path(int path);

/* Static description of a status code. */
const char *qlinear_status_string(int status);

#ifdef __cplusplus
}
#endif

#endif /* QLINEAR_H */
