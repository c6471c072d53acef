/*
 * Oracle for the block-quantized linear layer: a plain, slow, obviously
 * correct CPU implementation in fp64.
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
 * CPU-baseline leg of the benchmark may load this library.  The product
 * (the HIP library under paper_2607_08526_amd/) never links, includes or
 * calls anything here, and nothing here includes or calls the product.
 *
 * What it computes (paper: Methodology, "The aria runtime" and the
 * "Quantization and its evaluation" paragraph): the transformer's weights
 * are compressed to 8-bit or 4-bit integers (q8, q4) and the linear layers
 * are then evaluated from the compressed copy.  The paper fixes no format;
 * the format implemented here is the one the workload definitions give:
 * symmetric absmax, blocks of 32 consecutive weights along the reduction
 * dimension K, one fp16 scale per block, q4 codes packed two per byte.
 *
 * Readings taken where the paper is silent (each also listed in the design
 * notes of the repository):
 *   R1  Q = 127 for int8 and Q = 7 for q4 (symmetric; -128 and -8 are never
 *       produced, but are accepted as stored codes by the forward pass).
 *   R2  scale s = fp16 nearest to the exact quotient absmax / Q, ties to
 *       even, subnormals kept; a block whose rounded scale is not finite
 *       (absmax / Q >= 65520) is a range error, as is any NaN/Inf weight.
 *   R3  code c = clamp(nearest integer to the exact quotient w / s, ties to
 *       even, -Q, Q); a zero scale gives all-zero codes.
 *   R4  q4 packing: byte j of a row holds code 2j in its low nibble and
 *       code 2j+1 in its high nibble, both two's complement.
 *   R5  Y = X * W^T in fp64 from the stored codes and scales:
 *       Y[m][n] = sum_b s[n][b] * sum_{k in b} X[m][k] * c[n][k].
 *   R6  the unquantized reference (the fp16 weights the paper's table of
 *       precisions measures q8 / q4 against): Y = X * W^T in fp64 from fp16
 *       weight bit patterns W[N][K].
 *   R7  the epilogue a linear layer of a DiT block may carry (bias, the
 *       feed-forward's GELU, the residual add): Y = act(P + bias[n]) +
 *       residual[m][n] on the fp64 product P, act the identity or the GELU
 *       in its exact form x * Phi(x) = x * (1 + erf(x / sqrt 2)) / 2.
 *   R10 the self-attention around the linears (the GPU path's attention,
 *       Methodology; the fused attention the paper names as its open
 *       lever): per batch b, head h and query t,
 *       O[b,t,h,:] = sum_j p_j V[b,j,h,:] / sum_j p_j,
 *       p_j = exp(s_j - max_i s_i), s_j = scale * <Q[b,t,h,:], K[b,j,h,:]>,
 *       over all T keys of the same batch (no mask: the DiT attends
 *       bidirectionally); Q, K, V bf16 read from rows with strides.
 *   R9  steering (Methodology, additive injection, Eq. 2): the chosen
 *       block's output h gains alpha * ||h_bar|| * d for every token, d a
 *       unit direction [N], ||h_bar|| the layer's mean residual norm and
 *       alpha >= 0 the strength; alpha = 0 leaves h untouched.
 *   R8  W8A8 (the paper's 8-bit-arithmetic mode, Methodology and Table II:
 *       activations quantized alongside the weights, products in 8-bit
 *       integers).  The granularity is not stated; here one scale per
 *       token (row of X): s_x[m] = fp16 nearest to absmax_k |X[m][k]| / 127
 *       and q[m][k] = clamp(rint(X[m][k] / s_x[m]), -127, 127), i.e. R2 and
 *       R3 with the whole row as the block; int8 weights as R1-R3.  Then
 *       Y[m][n] = s_x[m] * sum_b s[n][b] * sum_{k in b} q[m][k] * c[n][k],
 *       each block's integer sum exact.
 *
 * Exactness of the arithmetic used for R2/R3 (why fp64 is enough):
 *   - absmax / Q: the fp64 quotient differs from the exact one by less than
 *     2^-53 relative, while a non-representable exact quotient lies at
 *     least ~2^-28 relative away from every fp16 rounding midpoint (absmax
 *     has 24 significant bits and Q < 2^7), so rounding the fp64 quotient
 *     to fp16 directly (never via fp32) equals rounding the exact quotient.
 *   - w / s: w has 24 and s 11 significant bits; a non-half-integer exact
 *     quotient lies at least 2^(e_w - e_s - 11) from every half-integer
 *     while the fp64 error is below 2^(e_w - e_s - 39), so rint() of the fp64
 *     quotient is the exact round-half-even integer.
 *
 * Precision: every arithmetic step is fp64; inputs (fp32 weights, bf16/fp32
 * activations, fp16 scales, integer codes) widen to fp64 exactly and every
 * product of two of them is exact in fp64.
 */
#include <math.h>
#include <stdint.h>
#include <string.h>

#define ORC_OK 0
#define ORC_ERR_INVALID 1
#define ORC_ERR_SHAPE 2
#define ORC_ERR_RANGE 4

#define ORC_FMT_Q4 4
#define ORC_FMT_INT8 8
#define ORC_DT_F32 0
#define ORC_DT_BF16 1

#define ORC_BLOCK 32

/* ---- number formats -------------------------------------------------- */

/* fp16 bit pattern of the value nearest to v, ties to even, subnormals
 * kept, overflow to +-inf (IEEE 754 binary16 rounding), done directly from
 * fp64 so that only one rounding happens. */
uint16_t oracle_f64_to_f16(double v)
{
    uint64_t bits;
    memcpy(&bits, &v, sizeof bits);
    uint16_t sign = (uint16_t)((bits >> 48) & 0x8000u);
    double a = fabs(v);
    if (isnan(v))
        return (uint16_t)(sign | 0x7E00u);
    /* 65520 is the midpoint between the largest finite fp16 (65504) and
     * 2^16; ties go to the even significand, which is 2^16, i.e. overflow. */
    if (a >= 65520.0)
        return (uint16_t)(sign | 0x7C00u);
    if (a < 0x1p-14) {
        /* subnormal range: a fixed quantum of 2^-24 */
        double q = rint(a * 0x1p24); /* scaling by 2^24 is exact */
        return (uint16_t)(sign | (uint16_t)q); /* q == 1024 encodes 2^-14 */
    }
    int e;
    (void)frexp(a, &e);                 /* a = f * 2^e, f in [0.5, 1) */
    int E = e - 1;                      /* a in [2^E, 2^(E+1)) */
    double q = rint(ldexp(a, 10 - E));  /* 11-bit significand, in [1024, 2048] */
    if (q == 2048.0) {                  /* rounded up into the next binade */
        q = 1024.0;
        E += 1;
    }
    return (uint16_t)(sign | (uint16_t)((E + 15) << 10) | (uint16_t)(q - 1024.0));
}

/* Exact value of an fp16 bit pattern. */
double oracle_f16_to_f64(uint16_t h)
{
    int sign = (h >> 15) & 1;
    int ex = (h >> 10) & 0x1F;
    int man = h & 0x3FF;
    double v;
    if (ex == 0)
        v = ldexp((double)man, -24);
    else if (ex == 31)
        v = man ? NAN : INFINITY;
    else
        v = ldexp((double)(man + 1024), ex - 25);
    return sign ? -v : v;
}

/* Exact value of a bf16 bit pattern (the upper half of an fp32). */
double oracle_bf16_to_f64(uint16_t b)
{
    uint32_t u = (uint32_t)b << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
}

/* ---- quantizer (R1-R4) ----------------------------------------------- */

static int qmax_of(int fmt)
{
    return fmt == ORC_FMT_INT8 ? 127 : 7;
}

/* Stored code at (row n, column k) as a signed integer. */
static int code_at(int fmt, const uint8_t *codes, int64_t K, int64_t n, int64_t k)
{
    if (fmt == ORC_FMT_INT8)
        return (int)(int8_t)codes[n * K + k];
    uint8_t byte = codes[n * (K / 2) + k / 2];
    int nib = (k & 1) ? (byte >> 4) : (byte & 0x0F);
    return nib >= 8 ? nib - 16 : nib;
}

static void store_code(int fmt, uint8_t *codes, int64_t K, int64_t n, int64_t k, int c)
{
    if (fmt == ORC_FMT_INT8) {
        codes[n * K + k] = (uint8_t)(int8_t)c;
        return;
    }
    uint8_t *p = &codes[n * (K / 2) + k / 2];
    uint8_t nib = (uint8_t)(c & 0x0F);
    if (k & 1)
        *p = (uint8_t)((*p & 0x0F) | (nib << 4));
    else
        *p = (uint8_t)((*p & 0xF0) | nib);
}

/* Quantize one block of 32 weights of row n.  Returns ORC_OK or
 * ORC_ERR_RANGE. */
static int quantize_block(int fmt, const float *w, int64_t K, int64_t n, int64_t b,
                          uint8_t *codes, uint16_t *scales)
{
    const int Q = qmax_of(fmt);
    double absmax = 0.0;
    for (int j = 0; j < ORC_BLOCK; ++j) {
        double v = (double)w[j];
        if (!isfinite(v))
            return ORC_ERR_RANGE;
        if (fabs(v) > absmax)
            absmax = fabs(v);
    }
    uint16_t sbits = oracle_f64_to_f16(absmax / (double)Q);
    if ((sbits & 0x7C00u) == 0x7C00u)
        return ORC_ERR_RANGE;
    scales[n * (K / ORC_BLOCK) + b] = sbits;
    double s = oracle_f16_to_f64(sbits);
    for (int j = 0; j < ORC_BLOCK; ++j) {
        int c = 0;
        if (s != 0.0) {
            double r = rint((double)w[j] / s);
            if (r > Q)
                r = Q;
            if (r < -Q)
                r = -Q;
            c = (int)r;
        }
        store_code(fmt, codes, K, n, b * ORC_BLOCK + j, c);
    }
    return ORC_OK;
}

/* W: fp32 [N][K] row-major; codes: int8 [N][K] or q4 [N][K/2]; scales: fp16
 * bits [N][K/32].  On ORC_ERR_RANGE the outputs are unspecified. */
int oracle_quantize(int fmt, const float *W, int64_t N, int64_t K,
                    uint8_t *codes, uint16_t *scales)
{
    if (fmt != ORC_FMT_INT8 && fmt != ORC_FMT_Q4)
        return ORC_ERR_INVALID;
    if (N <= 0 || K <= 0 || K % ORC_BLOCK)
        return ORC_ERR_SHAPE;
    if (!W || !codes || !scales)
        return ORC_ERR_INVALID;
    const int64_t nb = K / ORC_BLOCK;
    int status = ORC_OK;
#pragma omp parallel for schedule(static) reduction(|: status)
    for (int64_t n = 0; n < N; ++n)
        for (int64_t b = 0; b < nb; ++b)
            status |= quantize_block(fmt, W + n * K + b * ORC_BLOCK, K, n, b, codes, scales);
    return status ? ORC_ERR_RANGE : ORC_OK;
}

/* Wd[n][k] = c[n][k] * s[n][k/32] in fp64 (exact). */
int oracle_dequantize(int fmt, const uint8_t *codes, const uint16_t *scales,
                      int64_t N, int64_t K, double *Wd)
{
    if (fmt != ORC_FMT_INT8 && fmt != ORC_FMT_Q4)
        return ORC_ERR_INVALID;
    if (N <= 0 || K <= 0 || K % ORC_BLOCK)
        return ORC_ERR_SHAPE;
    for (int64_t n = 0; n < N; ++n)
        for (int64_t k = 0; k < K; ++k)
            Wd[n * K + k] = (double)code_at(fmt, codes, K, n, k) *
                            oracle_f16_to_f64(scales[n * (K / ORC_BLOCK) + k / ORC_BLOCK]);
    return ORC_OK;
}

/* ---- forward (R5) ---------------------------------------------------- */

static double x_at(const void *X, int xdt, int64_t K, int64_t m, int64_t k)
{
    if (xdt == ORC_DT_F32)
        return (double)((const float *)X)[m * K + k];
    return oracle_bf16_to_f64(((const uint16_t *)X)[m * K + k]);
}

static double output_element(int fmt, const void *X, int xdt, int64_t K,
                             const uint8_t *codes, const uint16_t *scales,
                             int64_t m, int64_t n)
{
    const int64_t nb = K / ORC_BLOCK;
    double y = 0.0;
    for (int64_t b = 0; b < nb; ++b) {
        double partial = 0.0;
        for (int j = 0; j < ORC_BLOCK; ++j) {
            int64_t k = b * ORC_BLOCK + j;
            partial += x_at(X, xdt, K, m, k) * (double)code_at(fmt, codes, K, n, k);
        }
        y += oracle_f16_to_f64(scales[n * nb + b]) * partial;
    }
    return y;
}

/* Y[m][n] for rows m = rows[0..nrows-1] of X (all n), written densely as
 * Y[i][n].  rows == NULL means rows 0..nrows-1.  X: [M][K] fp32 or bf16
 * bits; Y: fp64 [nrows][N]. */
int oracle_forward_rows(int fmt, const void *X, int xdt, int64_t M, int64_t K,
                        const uint8_t *codes, const uint16_t *scales, int64_t N,
                        const int64_t *rows, int64_t nrows, double *Y)
{
    if (fmt != ORC_FMT_INT8 && fmt != ORC_FMT_Q4)
        return ORC_ERR_INVALID;
    if (xdt != ORC_DT_F32 && xdt != ORC_DT_BF16)
        return ORC_ERR_INVALID;
    if (N <= 0 || K <= 0 || K % ORC_BLOCK || M < 0 || nrows < 0)
        return ORC_ERR_SHAPE;
    for (int64_t i = 0; i < nrows; ++i) {
        int64_t m = rows ? rows[i] : i;
        if (m < 0 || m >= M)
            return ORC_ERR_SHAPE;
    }
#pragma omp parallel for collapse(2) schedule(static)
    for (int64_t i = 0; i < nrows; ++i)
        for (int64_t n = 0; n < N; ++n)
            Y[i * N + n] = output_element(fmt, X, xdt, K, codes, scales,
                                          rows ? rows[i] : i, n);
    return ORC_OK;
}

/* Full product: Y fp64 [M][N]. */
int oracle_forward(int fmt, const void *X, int xdt, int64_t M, int64_t K,
                   const uint8_t *codes, const uint16_t *scales, int64_t N, double *Y)
{
    return oracle_forward_rows(fmt, X, xdt, M, K, codes, scales, N, NULL, M, Y);
}

/* ---- unquantized reference (R6) --------------------------------------- */

/* Y[i][n] = sum_k X[m][k] * W[n][k] for rows m = rows[i] (rows == NULL:
 * m = i), W fp16 bit patterns [N][K]; fp64. */
int oracle_forward_f16_rows(const void *X, int xdt, int64_t M, int64_t K, const uint16_t *W,
                            int64_t N, const int64_t *rows, int64_t nrows, double *Y)
{
    if (xdt != ORC_DT_F32 && xdt != ORC_DT_BF16)
        return ORC_ERR_INVALID;
    if (N <= 0 || K <= 0 || M < 0 || nrows < 0)
        return ORC_ERR_SHAPE;
    for (int64_t i = 0; i < nrows; ++i) {
        int64_t m = rows ? rows[i] : i;
        if (m < 0 || m >= M)
            return ORC_ERR_SHAPE;
    }
#pragma omp parallel for collapse(2) schedule(static)
    for (int64_t i = 0; i < nrows; ++i)
        for (int64_t n = 0; n < N; ++n) {
            const int64_t m = rows ? rows[i] : i;
            double y = 0.0;
            for (int64_t k = 0; k < K; ++k)
                y += x_at(X, xdt, K, m, k) * oracle_f16_to_f64(W[n * K + k]);
            Y[i * N + n] = y;
        }
    return ORC_OK;
}

/* ---- W8A8 (R8) ----------------------------------------------------------- */

/* Per-token int8 quantization of X [M][K] (fp32 or bf16 bits): q int8
 * [M][K], s fp16 bits [M].  ORC_ERR_RANGE for a non-finite activation or a
 * row whose rounded scale is not finite (the outputs are then unspecified). */
int oracle_quantize_act(const void *X, int xdt, int64_t M, int64_t K, int8_t *q, uint16_t *s)
{
    if (xdt != ORC_DT_F32 && xdt != ORC_DT_BF16)
        return ORC_ERR_INVALID;
    if (M < 0 || K <= 0)
        return ORC_ERR_SHAPE;
    int status = ORC_OK;
#pragma omp parallel for schedule(static) reduction(|: status)
    for (int64_t m = 0; m < M; ++m) {
        double absmax = 0.0;
        int bad = 0;
        for (int64_t k = 0; k < K; ++k) {
            const double v = x_at(X, xdt, K, m, k);
            if (!isfinite(v))
                bad = 1;
            else if (absmax < fabs(v))
                absmax = fabs(v);
        }
        const uint16_t sbits = oracle_f64_to_f16(absmax / 127.0);
        if (bad || (sbits & 0x7C00u) == 0x7C00u) {
            status |= ORC_ERR_RANGE;
            continue;
        }
        s[m] = sbits;
        const double sv = oracle_f16_to_f64(sbits);
        for (int64_t k = 0; k < K; ++k) {
            double r = sv != 0.0 ? rint(x_at(X, xdt, K, m, k) / sv) : 0.0;
            if (r > 127.0)
                r = 127.0;
            if (r < -127.0)
                r = -127.0;
            q[m * K + k] = (int8_t)r;
        }
    }
    return status ? ORC_ERR_RANGE : ORC_OK;
}

/* Y[i][n] (fp64) for rows m = rows[i] (rows == NULL: m = i) of the
 * quantized activations (qx [M][K], sx [M]) against int8 weights (codes
 * [N][K], scales [N][K/32]). */
int oracle_forward_w8a8_rows(const int8_t *qx, const uint16_t *sx, int64_t M, int64_t K,
                             const uint8_t *codes, const uint16_t *scales, int64_t N,
                             const int64_t *rows, int64_t nrows, double *Y)
{
    if (N <= 0 || K <= 0 || K % ORC_BLOCK || M < 0 || nrows < 0)
        return ORC_ERR_SHAPE;
    for (int64_t i = 0; i < nrows; ++i) {
        int64_t m = rows ? rows[i] : i;
        if (m < 0 || m >= M)
            return ORC_ERR_SHAPE;
    }
    const int64_t nb = K / ORC_BLOCK;
#pragma omp parallel for collapse(2) schedule(static)
    for (int64_t i = 0; i < nrows; ++i)
        for (int64_t n = 0; n < N; ++n) {
            const int64_t row = rows ? rows[i] : i;
            double y = 0.0;
            for (int64_t b = 0; b < nb; ++b) {
                int64_t dot = 0; /* exact: |dot| <= 32 * 127 * 128 */
                for (int j = 0; j < ORC_BLOCK; ++j) {
                    const int64_t k = b * ORC_BLOCK + j;
                    dot += (int64_t)qx[row * K + k] *
                           (int64_t)code_at(ORC_FMT_INT8, codes, K, n, k);
                }
                y += oracle_f16_to_f64(scales[n * nb + b]) * (double)dot;
            }
            Y[i * N + n] = oracle_f16_to_f64(sx[row]) * y;
        }
    return ORC_OK;
}

/* ---- epilogue (R7) ------------------------------------------------------ */

#define ORC_ACT_NONE 0
#define ORC_ACT_GELU 1

/* In place on Y[i][n] (fp64, nrows x N) holding the products of rows
 * m = rows[i] (rows == NULL: m = i): Y = act(Y + bias[n]) + residual[m][n];
 * bias [N] and residual [M][N] fp32, either may be NULL. */
int oracle_epilogue(double *Y, int64_t nrows, int64_t N, const int64_t *rows,
                    const float *bias, int act, const float *residual)
{
    if (act != ORC_ACT_NONE && act != ORC_ACT_GELU)
        return ORC_ERR_INVALID;
    if (N <= 0 || nrows < 0)
        return ORC_ERR_SHAPE;
    for (int64_t i = 0; i < nrows; ++i) {
        const int64_t src = rows ? rows[i] : i;  /* row of X, and of the residual */
        for (int64_t n = 0; n < N; ++n) {
            double v = Y[i * N + n];
            if (bias)
                v += (double)bias[n];
            if (act == ORC_ACT_GELU)
                v = v * 0.5 * (1.0 + erf(v / sqrt(2.0)));
            if (residual)
                v += (double)residual[src * N + n];
            Y[i * N + n] = v;
        }
    }
    return ORC_OK;
}

/* ---- steering (R9) ------------------------------------------------------ */

/* In place on Y (fp64, nrows x N): Y[i][n] += alpha * hnorm * dir[n], the
 * additive injection of Eq. 2; alpha == 0 leaves Y untouched. */
int oracle_steer(double *Y, int64_t nrows, int64_t N, const float *dir, double hnorm,
                 double alpha)
{
    if (N <= 0 || nrows < 0)
        return ORC_ERR_SHAPE;
    if (!dir)
        return ORC_ERR_INVALID;
    if (alpha == 0.0)
        return ORC_OK;
    const double c = alpha * hnorm;
    for (int64_t i = 0; i < nrows; ++i)
        for (int64_t n = 0; n < N; ++n)
            Y[i * N + n] += c * (double)dir[n];
    return ORC_OK;
}

/* ---- attention (R10) ----------------------------------------------------- */

/* O (fp64) for the listed query rows r = rows[i] = b * T + t (rows == NULL:
 * r = i) and every head: O[i][h * dh + c].  Q, K, V: bf16 bit patterns,
 * row r of Q at Q + r * ldq, head h at column h * dh (likewise K, V). */
int oracle_attention_rows(const uint16_t *Q, int64_t ldq, const uint16_t *K, int64_t ldk,
                          const uint16_t *V, int64_t ldv, int64_t B, int64_t T, int64_t H,
                          int64_t dh, double scale, const int64_t *rows, int64_t nrows, double *O)
{
    if (B <= 0 || T <= 0 || H <= 0 || dh <= 0 || nrows < 0)
        return ORC_ERR_SHAPE;
    if (!Q || !K || !V || !O)
        return ORC_ERR_INVALID;
    for (int64_t i = 0; i < nrows; ++i) {
        const int64_t r = rows ? rows[i] : i;
        if (r < 0 || r >= B * T)
            return ORC_ERR_SHAPE;
    }
#pragma omp parallel for collapse(2) schedule(static)
    for (int64_t i = 0; i < nrows; ++i)
        for (int64_t h = 0; h < H; ++h) {
            const int64_t r = rows ? rows[i] : i;
            const int64_t b = r / T;
            double smax = -INFINITY;
            for (int64_t j = 0; j < T; ++j) {
                double dot = 0.0;
                for (int64_t c = 0; c < dh; ++c)
                    dot += oracle_bf16_to_f64(Q[r * ldq + h * dh + c]) *
                           oracle_bf16_to_f64(K[(b * T + j) * ldk + h * dh + c]);
                if (scale * dot > smax)
                    smax = scale * dot;
            }
            double denom = 0.0;
            double *out = O + i * H * dh + h * dh;
            for (int64_t c = 0; c < dh; ++c)
                out[c] = 0.0;
            for (int64_t j = 0; j < T; ++j) {
                double dot = 0.0;
                for (int64_t c = 0; c < dh; ++c)
                    dot += oracle_bf16_to_f64(Q[r * ldq + h * dh + c]) *
                           oracle_bf16_to_f64(K[(b * T + j) * ldk + h * dh + c]);
                const double p = exp(scale * dot - smax);
                denom += p;
                for (int64_t c = 0; c < dh; ++c)
                    out[c] += p * oracle_bf16_to_f64(V[(b * T + j) * ldv + h * dh + c]);
            }
            for (int64_t c = 0; c < dh; ++c)
                out[c] /= denom;
        }
    return ORC_OK;
}

/* Number of threads the parallel loops above use (reported beside timings). */
#ifdef _OPENMP
#include <omp.h>
#endif
int oracle_num_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}
