// Quantized linear forward for few activation rows (bf16, M <= 64): the
// regime where the whole weight matrix is streamed once from HBM per call
// and time is set by HBM bandwidth, not by the matrix cores.
//
//   Y[m][n] = sum_b s[n][b] * sum_{k in b} X[m][k] * c[n][k]
//
// Decomposition.  A workgroup owns 16 weight rows (one MFMA column strip)
// and all M rows; its KW wavefronts split the K blocks between them and
// their fp32 partial outputs are summed through LDS in wavefront order, so
// the result is deterministic.  KW is chosen per shape so that the grid holds
// enough wavefronts to keep HBM busy even when N is small (N = 2048: 128
// workgroups of 8 wavefronts).
//
// Latency.  Every wavefront streams its codes, scales and activation
// fragments into registers D blocks ahead of use (loop unrolled by D, loads
// of the next D blocks issued before the current D are consumed).
//
// Contraction.  One v_mfma_f32_16x16x32_bf16 per block and 16-row activation
// subtile.  Codes enter the MFMA in offset form, exact in bf16 and cheap to
// build: int8 as byte ^ 0x80 = c + 128 (v_cvt_f32_ubyte), q4 as
// 0x4300 | (nibble ^ 8) = bf16(136 + c), two codes per AND-OR.  The offset's
// contribution -OFF * sum_{k in b} X[m][k] comes from a second MFMA of the
// same activation fragment against a constant -OFF matrix and enters the
// main MFMA as its C operand; the scale is then applied in fp32.  At these M
// the matrix cores are far from busy, so trading VALU work for an extra MFMA
// is the right exchange.  From M > 16 on (several row subtiles) the extra
// MFMA would cost more than it saves, and codes are converted exactly
// (sign-extended, then converted to fp32 and truncated to bf16).
#include <type_traits>

#include "epilogue.h"
#include "internal.h"

namespace qlk {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));


__device__ inline f32x4 mfma(u32x4 a, u32x4 b, f32x4 c)
{
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                   __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

__device__ inline uint32_t pack_hi(float lo, float hi)
{
    return __builtin_amdgcn_perm(__float_as_uint(hi), __float_as_uint(lo), 0x07060302u);
}

// int8 codes -> bf16 of c + 128 (natural k order)
__device__ inline u32x4 cvt_int8_off(uint2 c)
{
    const uint32_t a = c.x ^ 0x80808080u, b = c.y ^ 0x80808080u;
    u32x4 r;
    r[0] = pack_hi((float)(a & 0xFF), (float)((a >> 8) & 0xFF));
    r[1] = pack_hi((float)((a >> 16) & 0xFF), (float)(a >> 24));
    r[2] = pack_hi((float)(b & 0xFF), (float)((b >> 8) & 0xFF));
    r[3] = pack_hi((float)((b >> 16) & 0xFF), (float)(b >> 24));
    return r;
}

// q4 codes (one dword, k0 in bits 0-3) -> bf16 of c + 136 in the order
// (k0,k1), (k2,k3), (k4,k5), (k6,k7): byte j holds codes 2j (low nibble) and
// 2j+1; v_perm places byte j of x and of x >> 4 in the two 16-bit halves.
__device__ inline u32x4 cvt_q4_off(uint32_t c)
{
    const uint32_t x = c ^ 0x88888888u, y = x >> 4;
    u32x4 r;
    r[0] = (__builtin_amdgcn_perm(y, x, 0x0C040C00u) & 0x000F000Fu) | 0x43004300u;
    r[1] = (__builtin_amdgcn_perm(y, x, 0x0C050C01u) & 0x000F000Fu) | 0x43004300u;
    r[2] = (__builtin_amdgcn_perm(y, x, 0x0C060C02u) & 0x000F000Fu) | 0x43004300u;
    r[3] = (__builtin_amdgcn_perm(y, x, 0x0C070C03u) & 0x000F000Fu) | 0x43004300u;
    return r;
}

// Signed bit field [LO, LO + W) of x as a float (exact: |value| < 2^7).
template <int LO, int W>
__device__ inline float sfield(uint32_t x)
{
    return (float)((int32_t)(x << (32 - LO - W)) >> (32 - W));
}

__device__ inline u32x4 cvt_int8_exact(uint2 c)
{
    u32x4 r;
    r[0] = pack_hi(sfield<0, 8>(c.x), sfield<8, 8>(c.x));
    r[1] = pack_hi(sfield<16, 8>(c.x), sfield<24, 8>(c.x));
    r[2] = pack_hi(sfield<0, 8>(c.y), sfield<8, 8>(c.y));
    r[3] = pack_hi(sfield<16, 8>(c.y), sfield<24, 8>(c.y));
    return r;
}

__device__ inline u32x4 cvt_q4_exact(uint32_t c)
{
    u32x4 r;
    r[0] = pack_hi(sfield<0, 4>(c), sfield<4, 4>(c));
    r[1] = pack_hi(sfield<8, 4>(c), sfield<12, 4>(c));
    r[2] = pack_hi(sfield<16, 4>(c), sfield<20, 4>(c));
    r[3] = pack_hi(sfield<24, 4>(c), sfield<28, 4>(c));
    return r;
}

template <int FMT, int MSUB, int KW>
__global__ __launch_bounds__(64 * KW) void qgemm_skinny_kernel(const LinDesc d)
{
    constexpr bool OFFSET = MSUB == 1;                // offset-form codes + correction MFMA
    constexpr int D = MSUB >= 4 ? 2 : MSUB == 2 ? 4 : 8;  // blocks in flight per buffer
    typedef typename std::conditional<FMT == QL_FMT_INT8, uint2, uint32_t>::type CodeT;

    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int l16 = lane & 15, lg = lane >> 4;
    const int M = d.M, N = d.N, K = d.K, nb = K >> 5;
    const int n0 = (int)blockIdx.x * 16;
    const int row = min(n0 + l16, N - 1);

    // this wavefront's blocks [b_beg, b_end)
    const int per = (nb + KW - 1) / KW;
    const int b_beg = min(wave * per, nb), b_end = min(b_beg + per, nb);

    const uint8_t *crow = d.codes + (int64_t)row * (FMT == QL_FMT_INT8 ? K : K / 2) +
                          (FMT == QL_FMT_INT8 ? lg * 8 : lg * 4);
    const uint16_t *srow = d.scales + (int64_t)row * nb;
    const uint16_t *xrow[MSUB];
#pragma unroll
    for (int i = 0; i < MSUB; ++i)
        xrow[i] = reinterpret_cast<const uint16_t *>(d.X) +
                  (int64_t)min(i * 16 + l16, M - 1) * K + lg * 8;

    // constant -OFF matrix (bf16), for the offset correction
    const uint32_t negoff = FMT == QL_FMT_INT8 ? 0xC300C300u : 0xC308C308u;  // -128 / -136
    const u32x4 bneg = {negoff, negoff, negoff, negoff};

    f32x4 acc[MSUB];
#pragma unroll
    for (int i = 0; i < MSUB; ++i)
        acc[i] = f32x4{0.f, 0.f, 0.f, 0.f};

    CodeT cb[2][D];
    uint32_t sb[2][D];
    u32x4 xb[2][D][MSUB];

    auto load = [&](int buf, int b0) {
#pragma unroll
        for (int t = 0; t < D; ++t) {
            const int b = min(b0 + t, nb - 1);  // past the end: a valid, unused block
            cb[buf][t] = *reinterpret_cast<const CodeT *>(crow + (int64_t)b * (FMT == QL_FMT_INT8 ? 32 : 16));
            sb[buf][t] = srow[b];
#pragma unroll
            for (int i = 0; i < MSUB; ++i)
                xb[buf][t][i] = *reinterpret_cast<const u32x4 *>(xrow[i] + (int64_t)b * 32);
        }
    };
    auto compute = [&](int buf, int b0) {
#pragma unroll
        for (int t = 0; t < D; ++t) {
            if (b0 + t < b_end) {
                u32x4 B;
                if (OFFSET)
                    B = FMT == QL_FMT_INT8 ? cvt_int8_off(*(uint2 *)&cb[buf][t])
                                           : cvt_q4_off(*(uint32_t *)&cb[buf][t]);
                else
                    B = FMT == QL_FMT_INT8 ? cvt_int8_exact(*(uint2 *)&cb[buf][t])
                                           : cvt_q4_exact(*(uint32_t *)&cb[buf][t]);
                const float s = (float)__builtin_bit_cast(_Float16, (uint16_t)sb[buf][t]);
#pragma unroll
                for (int i = 0; i < MSUB; ++i) {
                    f32x4 T = {0.f, 0.f, 0.f, 0.f};
                    if (OFFSET)
                        T = mfma(xb[buf][t][i], bneg, T);
                    acc[i] += s * mfma(xb[buf][t][i], B, T);
                }
            }
        }
    };

    if (b_beg < b_end) {
        load(0, b_beg);
        for (int b0 = b_beg; b0 < b_end; b0 += 2 * D) {
            if (b0 + D < b_end)
                load(1, b0 + D);
            compute(0, b0);
            if (b0 + 2 * D < b_end)
                load(0, b0 + 2 * D);
            if (b0 + D < b_end)
                compute(1, b0 + D);
        }
    }

    // sum the wavefronts' partial outputs in wavefront order
    __shared__ __align__(16) float red[KW][MSUB][64][4];
#pragma unroll
    for (int i = 0; i < MSUB; ++i)
        *reinterpret_cast<f32x4 *>(&red[wave][i][lane][0]) = acc[i];
    __syncthreads();
    if (wave == 0) {
#pragma unroll
        for (int i = 0; i < MSUB; ++i) {
            f32x4 y = *reinterpret_cast<const f32x4 *>(&red[0][i][lane][0]);
#pragma unroll
            for (int w = 1; w < KW; ++w)
                y += *reinterpret_cast<const f32x4 *>(&red[w][i][lane][0]);
            const int n = n0 + l16;
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int m = i * 16 + lg * 4 + r;
                if (m < M && n < N)
                    epi_store(d.ep, d.Y, (int64_t)m * N + n, n, y[r]);
            }
        }
    }
}

template <int FMT, int MSUB>
hipError_t launch_ms(int kw, const LinDesc &d, hipStream_t s)
{
    const dim3 grid((unsigned)((d.N + 15) / 16));
    switch (kw) {
    case 4:
        hipLaunchKernelGGL((qgemm_skinny_kernel<FMT, MSUB, 4>), grid, dim3(256), 0, s, d);
        break;
    case 8:
        hipLaunchKernelGGL((qgemm_skinny_kernel<FMT, MSUB, 8>), grid, dim3(512), 0, s, d);
        break;
    default:
        return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

}  // namespace

int skinny_max_m() { return 64; }

hipError_t launch_qgemm_skinny(int fmt, const LinDesc &d, hipStream_t stream)
{
    // wavefronts per workgroup: enough that the grid holds ~2048 wavefronts,
    // without giving a wavefront fewer than 8 blocks
    const int groups = (d.N + 15) / 16;
    const int nb = d.K / 32;
    // (at most 8: 1024-thread workgroups leave 128 VGPRs per lane, too few
    // for the load window)
    int kw = 4;
    if (groups * kw < 2048 && nb / 8 >= 8)
        kw = 8;
    if (fmt == QL_FMT_INT8)
        return d.M <= 16   ? launch_ms<QL_FMT_INT8, 1>(kw, d, stream)
               : d.M <= 32 ? launch_ms<QL_FMT_INT8, 2>(kw, d, stream)
                           : launch_ms<QL_FMT_INT8, 4>(kw, d, stream);
    return d.M <= 16   ? launch_ms<QL_FMT_Q4, 1>(kw, d, stream)
           : d.M <= 32 ? launch_ms<QL_FMT_Q4, 2>(kw, d, stream)
                       : launch_ms<QL_FMT_Q4, 4>(kw, d, stream);
}

}  // namespace qlk
