// Block quantizer: fp32 weights -> int8 or 4-bit codes + fp16 scales.
//
// Paper (Methodology, "Quantization and its evaluation"): the transformer's
// weights are compressed to 8-bit or 4-bit integers; the compressed copy then
// replaces the full-precision one.  Encoding used here: symmetric absmax over
// blocks of 32 weights along K, scale = fp16 nearest to absmax / Q (one
// rounding of the exact quotient, ties to even), code = nearest integer to
// w / scale (ties to even) clamped to [-Q, Q]; Q = 127 (int8) or 7 (q4).
//
// Exactness: the quotients are formed in fp64 (w has 24 and the scale 11
// significant bits, Q < 2^7), which keeps every rounding decision identical
// to rounding the exact real quotient; fp64 -> fp16 is converted directly
// from the fp64 bit pattern with integer arithmetic, never through fp32.
//
// Layout: 4 lanes per 32-weight block, 8 consecutive weights per lane (two
// 16-byte loads); the 4 lanes of a block are adjacent in a wavefront and
// combine their absmax with two butterfly shuffles.
#include "internal.h"

namespace qlk {
namespace {

// fp16 bit pattern nearest to the non-negative finite double q (ties to
// even significand, subnormals kept, 0x7C00 when it rounds past 65504).
__device__ inline uint32_t f64_to_f16_bits(double q)
{
    const uint64_t u = (uint64_t)__double_as_longlong(q);
    const int ebits = (int)((u >> 52) & 0x7FF);
    if (ebits == 0)
        return 0;  // zero or an fp64 subnormal: far below half the fp16 quantum
    const int E = ebits - 1023;                       // q in [2^E, 2^(E+1))
    const uint64_t sig = (u & 0xFFFFFFFFFFFFFull) | (1ull << 52);  // 53 bits
    if (E >= 16)
        return 0x7C00;
    if (E >= -14) {
        // normal fp16: keep 11 significant bits
        uint64_t keep = sig >> 42;
        const uint64_t rem = sig & ((1ull << 42) - 1);
        const uint64_t half = 1ull << 41;
        if (rem > half || (rem == half && (keep & 1)))
            ++keep;
        int e = E;
        if (keep == 2048) {
            keep = 1024;
            ++e;
        }
        if (e >= 16)
            return 0x7C00;
        return (uint32_t)(((e + 15) << 10) | (int)(keep - 1024));
    }
    // fp16 subnormal range: value / 2^-24 = sig * 2^(E - 28)
    const int sh = 28 - E;  // >= 43
    if (sh > 63)
        return 0;  // below 2^-36, under half a quantum
    uint64_t keep = sig >> sh;
    const uint64_t rem = sig & ((1ull << sh) - 1);
    const uint64_t half = 1ull << (sh - 1);
    if (rem > half || (rem == half && (keep & 1)))
        ++keep;
    return (uint32_t)keep;  // 1024 encodes 2^-14, the smallest normal
}

// Exact value of a finite fp16 bit pattern with the sign bit clear.
__device__ inline double f16_bits_to_f64(uint32_t h)
{
    const uint32_t ex = (h >> 10) & 0x1F;
    const uint32_t man = h & 0x3FF;
    if (ex == 0)
        return (double)man * 0x1p-24;
    const uint64_t bits = ((uint64_t)(ex - 15 + 1023) << 52) | ((uint64_t)man << 42);
    return __longlong_as_double((long long)bits);
}

template <int FMT>
__global__ __launch_bounds__(256) void quantize_kernel(const float *__restrict__ W,
                                                       int64_t n_blocks,
                                                       uint8_t *__restrict__ codes,
                                                       uint16_t *__restrict__ scales,
                                                       int *__restrict__ status)
{
    constexpr int Q = FMT == QL_FMT_INT8 ? 127 : 7;
    const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
    const int64_t blk = t >> 2;  // row-major block index n * (K/32) + b
    const int part = (int)(t & 3);
    const bool valid = blk < n_blocks;

    uint32_t wb[8];
    if (valid) {
        const uint4 *p = reinterpret_cast<const uint4 *>(W + blk * 32 + part * 8);
        const uint4 a = p[0], b = p[1];
        wb[0] = a.x; wb[1] = a.y; wb[2] = a.z; wb[3] = a.w;
        wb[4] = b.x; wb[5] = b.y; wb[6] = b.z; wb[7] = b.w;
    } else {
#pragma unroll
        for (int j = 0; j < 8; ++j)
            wb[j] = 0;
    }

    // |w| compared as unsigned integers (monotone for non-NaN fp32 bit
    // patterns); anything at or above the +inf pattern is a NaN or Inf.
    uint32_t amax = 0;
    bool bad = false;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        const uint32_t a = wb[j] & 0x7FFFFFFFu;
        bad |= a >= 0x7F800000u;
        amax = a > amax ? a : amax;
    }
    {
        const uint32_t o1 = (uint32_t)__shfl_xor((int)amax, 1);
        amax = o1 > amax ? o1 : amax;
        const uint32_t o2 = (uint32_t)__shfl_xor((int)amax, 2);
        amax = o2 > amax ? o2 : amax;
    }
    if (!valid)
        return;
    if (amax >= 0x7F800000u) {  // some lane of this block saw a NaN/Inf
        if (bad)
            *status = QL_ERR_RANGE;
        return;
    }

    const double a = (double)__uint_as_float(amax);
    const uint32_t sbits = f64_to_f16_bits(a / (double)Q);
    if (sbits == 0x7C00) {
        if (part == 0)
            *status = QL_ERR_RANGE;
        return;
    }
    const double s = f16_bits_to_f64(sbits);

    int c[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        int v = 0;
        if (s != 0.0) {
            double r = rint((double)__uint_as_float(wb[j]) / s);
            r = r > (double)Q ? (double)Q : r;
            r = r < -(double)Q ? -(double)Q : r;
            v = (int)r;
        }
        c[j] = v;
    }

    if (part == 0)
        scales[blk] = (uint16_t)sbits;
    if (FMT == QL_FMT_INT8) {
        uint32_t lo = 0, hi = 0;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            lo |= (uint32_t)(c[j] & 0xFF) << (8 * j);
            hi |= (uint32_t)(c[j + 4] & 0xFF) << (8 * j);
        }
        *reinterpret_cast<uint2 *>(codes + blk * 32 + part * 8) = make_uint2(lo, hi);
    } else {
        uint32_t word = 0;
#pragma unroll
        for (int j = 0; j < 8; ++j)
            word |= (uint32_t)(c[j] & 0xF) << (4 * j);
        *reinterpret_cast<uint32_t *>(codes + blk * 16 + part * 4) = word;
    }
}

// Per-token activation quantizer of the W8A8 path: one workgroup per row of
// X.  Scale = fp16 nearest to (row absmax) / 127 and code = nearest integer
// to x / scale clamped to [-127, 127] (the weight rules with the whole row as
// the block).  bf16 activations have 8 significant bits, so a correctly
// rounded fp32 quotient already decides every rounding as the exact one
// would (a non-half-integer quotient lies at least 2^-9 of its size from
// every half-integer, the fp32 error is below 2^-24 of it, and exact
// half-integers are representable); fp32 activations use fp64 as the
// weight quantizer does.  A row holding a NaN or Inf, or whose scale would
// overflow fp16, gets the NaN scale 0x7E00 and zero codes, so its outputs
// come out NaN.
template <bool BF16>
__device__ inline void load8(const void *X, int64_t e, uint32_t (&v)[8])
{
    if constexpr (BF16) {
        const uint4 a = *reinterpret_cast<const uint4 *>(static_cast<const uint16_t *>(X) + e);
        const uint32_t w[4] = {a.x, a.y, a.z, a.w};
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            v[2 * j] = w[j] << 16;
            v[2 * j + 1] = w[j] & 0xFFFF0000u;
        }
    } else {
        const uint4 *p = reinterpret_cast<const uint4 *>(static_cast<const float *>(X) + e);
        const uint4 a = p[0], b = p[1];
        v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
        v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
    }
}

template <bool BF16>
__global__ __launch_bounds__(256) void act_quant_kernel(const void *__restrict__ X, int64_t K,
                                                        int8_t *__restrict__ q,
                                                        uint16_t *__restrict__ sx)
{
    __shared__ uint32_t wmax[4];
    const int64_t row = (int64_t)blockIdx.x * K;
    const int tid = threadIdx.x;
    const int64_t groups = K / 8;
    uint32_t amax = 0;  // |x| bit patterns compare like the values; NaN/Inf >= 0x7F800000
    for (int64_t g = tid; g < groups; g += 256) {
        uint32_t v[8];
        load8<BF16>(X, row + 8 * g, v);
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const uint32_t a = v[j] & 0x7FFFFFFFu;
            amax = a > amax ? a : amax;
        }
    }
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const uint32_t t = (uint32_t)__shfl_xor((int)amax, o);
        amax = t > amax ? t : amax;
    }
    if ((tid & 63) == 0)
        wmax[tid >> 6] = amax;
    __syncthreads();
    amax = wmax[0];
#pragma unroll
    for (int w = 1; w < 4; ++w)
        amax = wmax[w] > amax ? wmax[w] : amax;

    uint32_t sbits = 0x7C00;
    if (amax < 0x7F800000u)
        sbits = f64_to_f16_bits((double)__uint_as_float(amax) / 127.0);
    const bool bad = sbits == 0x7C00;
    if (tid == 0)
        sx[blockIdx.x] = (uint16_t)(bad ? 0x7E00 : sbits);
    const double sd = f16_bits_to_f64(sbits);
    const float sf = (float)sd;  // exact: an fp16 value
    for (int64_t g = tid; g < groups; g += 256) {
        uint32_t v[8];
        load8<BF16>(X, row + 8 * g, v);
        int c[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            int r = 0;
            if (!bad && sbits != 0) {
                const float x = __uint_as_float(v[j]);
                float t;
                if constexpr (BF16)
                    t = rintf(__fdiv_rn(x, sf));
                else
                    t = (float)rint((double)x / sd);
                t = t > 127.0f ? 127.0f : t;
                t = t < -127.0f ? -127.0f : t;
                r = (int)t;
            }
            c[j] = r;
        }
        uint32_t lo = 0, hi = 0;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            lo |= (uint32_t)(c[j] & 0xFF) << (8 * j);
            hi |= (uint32_t)(c[j + 4] & 0xFF) << (8 * j);
        }
        *reinterpret_cast<uint2 *>(q + row + 8 * g) = make_uint2(lo, hi);
    }
}

}  // namespace

hipError_t launch_act_quant(const void *X, bool bf16, int64_t M, int64_t K, int8_t *q,
                            uint16_t *sx, hipStream_t stream)
{
    if (bf16)
        hipLaunchKernelGGL(act_quant_kernel<true>, dim3((unsigned)M), dim3(256), 0, stream, X, K,
                           q, sx);
    else
        hipLaunchKernelGGL(act_quant_kernel<false>, dim3((unsigned)M), dim3(256), 0, stream, X,
                           K, q, sx);
    return hipGetLastError();
}

hipError_t launch_quantize(int fmt, const float *W, int64_t N, int64_t K, uint8_t *codes,
                           uint16_t *scales, int *status, hipStream_t stream)
{
    const int64_t n_blocks = N * (K / 32);
    const int64_t threads = n_blocks * 4;
    const int64_t grid = (threads + 255) / 256;
    if (fmt == QL_FMT_INT8)
        hipLaunchKernelGGL(quantize_kernel<QL_FMT_INT8>, dim3((unsigned)grid), dim3(256), 0,
                           stream, W, n_blocks, codes, scales, status);
    else
        hipLaunchKernelGGL(quantize_kernel<QL_FMT_Q4>, dim3((unsigned)grid), dim3(256), 0,
                           stream, W, n_blocks, codes, scales, status);
    return hipGetLastError();
}

}  // namespace qlk
