// Activation pre-pass of the large-M forward: bf16 X [M][K] -> fp16 X' [M][K]
// with a per-row power-of-two shift e[m], X'[m][k] = X[m][k] * 2^-e[m].
//
// bf16 carries 8 significant bits and fp16 11, so the conversion is exact
// whenever the shifted value lands in fp16's normal range.  e[m] puts the
// row's largest magnitude in [2^14, 2^15): nothing overflows, and only values
// below 2^-29 of the row maximum (fp16 subnormals after the shift) are
// rounded, by at most 2^-25 of the shifted scale.  The forward kernel
// multiplies its fp32 results back by 2^e[m] exactly.
//
// One wavefront per row (four rows per workgroup), the rows of every
// activation tensor of a call in one launch; rows up to 16384 wide are read
// once into the wavefront's registers (16-byte chunks, lane l taking chunks
// l, l + 64, ...), reduced to the row maximum by lane exchanges (no
// barrier), then converted and stored.  Wider rows take one workgroup per
// row and two passes.  For the q4 kernel each 8-k group is stored in the
// slot order of its weight conversion (qgemm_wide.hip).
#include "internal.h"

namespace qlk {
namespace {

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__device__ inline uint32_t bf16_absmax2(uint32_t v)
{
    return max(v & 0x7FFFu, (v >> 16) & 0x7FFFu);
}

// the shift e of a row whose largest |x| has the bf16 bit pattern mx:
// exponent of the row maximum (bf16: value in [2^(E-127), 2^(E-126)));
// zero, subnormal-only or non-finite rows keep e = 0
__device__ inline int shift_of(uint32_t mx)
{
    const int E = (int)(mx >> 7);
    return (E >= 1 && E <= 254) ? (E - 127) - 14 : 0;
}

// largest |x| of the row, compared as bf16 bit patterns (monotone for
// non-NaN magnitudes), reduced over the workgroup -> the row's shift e
__device__ inline int row_shift(uint32_t mx, int *rexp, int m)
{
    __shared__ uint32_t wmax[4];
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1)
        mx = max(mx, (uint32_t)__shfl_xor((int)mx, o));
    if ((threadIdx.x & 63) == 0)
        wmax[threadIdx.x >> 6] = mx;
    __syncthreads();
    mx = max(max(wmax[0], wmax[1]), max(wmax[2], wmax[3]));
    const int e = shift_of(mx);
    if (threadIdx.x == 0)
        rexp[m] = e;
    return e;
}

// 8 bf16 (k0..k7) -> 8 fp16 of X * 2^-e, in natural order, or (SLOTS) in the
// slot order of the q4 weight conversion: position e holds k = Q4_SLOT[e]
template <bool SLOTS>
__device__ inline u32x4 to_f16(u32x4 v, int e)
{
    half8 h;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        h[2 * j] = (_Float16)__builtin_amdgcn_ldexpf(__uint_as_float(v[j] << 16), -e);
        h[2 * j + 1] = (_Float16)__builtin_amdgcn_ldexpf(__uint_as_float(v[j] & 0xFFFF0000u), -e);
    }
    if constexpr (SLOTS) {
        half8 p;
#pragma unroll
        for (int i = 0; i < 8; ++i)
            p[i] = h[Q4_SLOT[i]];
        h = p;
    }
    return __builtin_bit_cast(u32x4, h);
}

// C chunks of 16 bytes per lane (K / 8 <= 64 C): wavefront w of workgroup
// b converts global row 4 b + w, i.e. row r - row_begin[i] of job i (all
// activation tensors of a call in one launch, rows numbered consecutively).
template <int C, bool SLOTS>
__global__ __launch_bounds__(256) void xprep_wave_kernel(const XprepArgs a, int rows,
                                                         int *__restrict__ zero, int nzero)
{
    if (blockIdx.x == 0)
        for (int i = threadIdx.x; i < nzero; i += 256)
            zero[i] = 0;
    const int r = (int)blockIdx.x * 4 + (int)(threadIdx.x >> 6), lane = threadIdx.x & 63;
    if (r >= rows)
        return;  // the whole wavefront
    int ji = 0;
#pragma unroll
    for (int i = 1; i < QL_MAX_GROUP; ++i)
        if (i < a.n && r >= a.row_begin[i])
            ji = i;
    const XprepJob &jb = a.j[ji];
    const int m = r - a.row_begin[ji], K = jb.K, n16 = K / 8;
    const u32x4 *row = reinterpret_cast<const u32x4 *>(reinterpret_cast<const uint16_t *>(jb.X) +
                                                       (int64_t)m * K);
    u32x4 *out = reinterpret_cast<u32x4 *>(jb.Xh + (int64_t)m * K);
    u32x4 v[C];
    uint32_t mx = 0;
#pragma unroll
    for (int c = 0; c < C; ++c) {
        const int i = lane + 64 * c;
        v[c] = i < n16 ? row[i] : u32x4{0u, 0u, 0u, 0u};
#pragma unroll
        for (int j = 0; j < 4; ++j)
            mx = max(mx, bf16_absmax2(v[c][j]));
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1)
        mx = max(mx, (uint32_t)__shfl_xor((int)mx, o));
    const int e = shift_of(mx);
    if (lane == 0)
        jb.rexp[m] = e;
#pragma unroll
    for (int c = 0; c < C; ++c) {
        const int i = lane + 64 * c;
        if (i < n16)
            out[i] = to_f16<SLOTS>(v[c], e);
    }
}

// Rows wider than 16384: one workgroup per row, a max pass and a convert
// pass (the second read of the row hits L2).  Workgroup b converts row
// b - row_begin[i] of job i.
template <bool SLOTS>
__global__ __launch_bounds__(256) void xprep_row_kernel(const XprepArgs a, int *__restrict__ zero,
                                                        int nzero)
{
    const int b = blockIdx.x;
    if (b == 0)
        for (int i = threadIdx.x; i < nzero; i += 256)
            zero[i] = 0;
    int ji = 0;
#pragma unroll
    for (int i = 1; i < QL_MAX_GROUP; ++i)
        if (i < a.n && b >= a.row_begin[i])
            ji = i;
    const XprepJob &jb = a.j[ji];
    const int m = b - a.row_begin[ji], K = jb.K;
    const uint16_t *X = reinterpret_cast<const uint16_t *>(jb.X);
    const u32x4 *row = reinterpret_cast<const u32x4 *>(X + (int64_t)m * K);
    u32x4 *out = reinterpret_cast<u32x4 *>(jb.Xh + (int64_t)m * K);
    const int n16 = K / 8;
    uint32_t mx = 0;
    for (int i = threadIdx.x; i < n16; i += 256) {
        const u32x4 v = row[i];
#pragma unroll
        for (int j = 0; j < 4; ++j)
            mx = max(mx, bf16_absmax2(v[j]));
    }
    const int e = row_shift(mx, jb.rexp, m);
    for (int i = threadIdx.x; i < n16; i += 256)
        out[i] = to_f16<SLOTS>(row[i], e);
}

template <bool SLOTS>
void launch_xprep_t(const XprepArgs &a, int rows, int maxK, int *zero, int nzero,
                    hipStream_t stream)
{
    const int n16 = maxK / 8;
    const dim3 block(256), wgrid((unsigned)((rows + 3) / 4));
    if (n16 <= 64 * 4)
        hipLaunchKernelGGL((xprep_wave_kernel<4, SLOTS>), wgrid, block, 0, stream, a, rows, zero,
                           nzero);
    else if (n16 <= 64 * 8)
        hipLaunchKernelGGL((xprep_wave_kernel<8, SLOTS>), wgrid, block, 0, stream, a, rows, zero,
                           nzero);
    else if (n16 <= 64 * 16)
        hipLaunchKernelGGL((xprep_wave_kernel<16, SLOTS>), wgrid, block, 0, stream, a, rows, zero,
                           nzero);
    else if (n16 <= 64 * 32)
        hipLaunchKernelGGL((xprep_wave_kernel<32, SLOTS>), wgrid, block, 0, stream, a, rows, zero,
                           nzero);
    else
        hipLaunchKernelGGL((xprep_row_kernel<SLOTS>), dim3((unsigned)rows), block, 0, stream, a,
                           zero, nzero);
}

}  // namespace

hipError_t launch_xprep(const XprepJob *jobs, int n, bool q4_slots, int *zero, int nzero,
                        hipStream_t stream)
{
    XprepArgs a{};
    int rows = 0, maxK = 0;
    for (int i = 0; i < n; ++i) {
        a.j[i] = jobs[i];
        a.row_begin[i] = rows;
        rows += jobs[i].M;
        maxK = jobs[i].K > maxK ? jobs[i].K : maxK;
    }
    a.n = n;
    if (q4_slots)
        launch_xprep_t<true>(a, rows, maxK, zero, nzero, stream);
    else
        launch_xprep_t<false>(a, rows, maxK, zero, nzero, stream);
    return hipGetLastError();
}

}  // namespace qlk
