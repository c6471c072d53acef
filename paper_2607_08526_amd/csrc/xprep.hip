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
//
// The same launch sets the weight-row shifts of the int8 / q4 layers (one
// wavefront per K part and weight row): the forward kernel's tiles then
// read one shift per row instead of scanning the row's scales, every row
// tile again.
#include <algorithm>

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

// The shifts f of eight (K part p, weight row n) items, one per group of 8
// lanes: the largest scale of the part's blocks (16-byte chunks of 8
// scales, lane l of the group taking chunks l, l + 8, ...; fp16 bit
// patterns of non-negative values order as integers, the sign bit is
// ignored), reduced by lane exchanges within the group; then qmax * smax *
// 2^f lies in [2^14, 2^15), so that every |c * s * 2^f| of the part is below
// 2^15.  The part's blocks are whole 16-byte chunks (K % 256 == 0, parts of
// whole scale groups) and the scales 16-byte aligned.  Item t (numbered
// over all jobs, part-major within a job) of the calling lane's group.
__device__ inline void weight_shifts(const XprepArgs &a, int64_t t, int64_t items, int lane)
{
    const bool live = t < items;
    int ji = 0;
#pragma unroll
    for (int i = 1; i < QL_MAX_GROUP; ++i)
        if (i < a.nw && t >= a.wrow_begin[i])
            ji = i;
    const WshiftJob &w = a.w[ji];
    const int u = live ? (int)(t - a.wrow_begin[ji]) : 0;
    const int p = u / w.ld, n = u - p * w.ld, sub = lane & 7;
    const int b0 = p * w.pblocks, b1 = min(b0 + w.pblocks, w.nb);
    const u32x4 *row =
        reinterpret_cast<const u32x4 *>(w.scales + (int64_t)min(n, w.N - 1) * w.nb);
    uint32_t mx = 0;
    if (live)
#pragma unroll 4
        for (int q = b0 / 8 + sub; q < b1 / 8; q += 8) {
            const u32x4 v = row[q];
#pragma unroll
            for (int j = 0; j < 4; ++j)
                mx = max(mx, max(v[j] & 0x7FFFu, (v[j] >> 16) & 0x7FFFu));
        }
#pragma unroll
    for (int o = 4; o >= 1; o >>= 1)
        mx = max(mx, (uint32_t)__shfl_xor((int)mx, o));
    if (live && sub == 0) {
        const float smax = (float)__builtin_bit_cast(_Float16, (uint16_t)mx);
        int E = 0;
        (void)__builtin_frexpf(smax * (float)w.qmax, &E);
        w.f[p * w.ld + n] = mx ? 15 - E : 0;
    }
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

// Row r of the activation jobs by one wavefront (C chunks of 16 bytes per
// lane): the row maximum by lane exchanges, the shift, the conversion.
template <int C, bool SLOTS>
__device__ inline void convert_row(const XprepArgs &a, int r, int lane)
{
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


// C chunks of 16 bytes per lane (K / 8 <= 64 C): wavefront w of workgroup
// b converts global row r = 4 b + w, i.e. row r - row_begin[i] of job i
// (all activation tensors of a call in one launch, rows numbered
// consecutively), then sets the weight-row shifts of items 8 r .. 8 r + 7
// (latency-bound reads that ride on the row streaming; the grid covers
// the larger of the two counts).
template <int C, bool SLOTS>
__global__ __launch_bounds__(256) void xprep_wave_kernel(const XprepArgs a, int rows, int witems,
                                                         int *__restrict__ zero, int nzero)
{
    if (blockIdx.x == 0)
        for (int i = threadIdx.x; i < nzero; i += 256)
            zero[i] = 0;
    const int r = (int)blockIdx.x * 4 + (int)(threadIdx.x >> 6), lane = threadIdx.x & 63;
    if (r < rows)
        convert_row<C, SLOTS>(a, r, lane);
    if ((int64_t)r * 8 < witems)  // the whole wavefront
        weight_shifts(a, (int64_t)r * 8 + lane / 8, witems, lane);
}

// Rows wider than 16384: one workgroup per row, a max pass and a convert
// pass (the second read of the row hits L2).  Workgroup b sets the
// weight-row shifts of items 32 b .. 32 b + 31 and converts row b -
// row_begin[i] of job i (the grid covers the larger of the two counts).
template <bool SLOTS>
__global__ __launch_bounds__(256) void xprep_row_kernel(const XprepArgs a, int rows, int witems,
                                                        int *__restrict__ zero, int nzero)
{
    const int b = blockIdx.x;
    if (b == 0)
        for (int i = threadIdx.x; i < nzero; i += 256)
            zero[i] = 0;
    const int64_t t = (int64_t)b * 32 + threadIdx.x / 8;  // four batches of 8 items
    if (t - threadIdx.x % 64 / 8 < witems)               // the whole wavefront
        weight_shifts(a, t, witems, threadIdx.x & 63);
    if (b >= rows)
        return;
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
void launch_xprep_t(const XprepArgs &a, int rows, int witems, int maxK, int *zero, int nzero,
                    hipStream_t stream)
{
    const int n16 = maxK / 8;
    const int64_t waves = std::max<int64_t>(rows, (witems + 7) / 8);
    const dim3 block(256), wgrid((unsigned)((waves + 3) / 4));
    if (n16 <= 64 * 4)
        hipLaunchKernelGGL((xprep_wave_kernel<4, SLOTS>), wgrid, block, 0, stream, a, rows, witems,
                           zero, nzero);
    else if (n16 <= 64 * 8)
        hipLaunchKernelGGL((xprep_wave_kernel<8, SLOTS>), wgrid, block, 0, stream, a, rows, witems,
                           zero, nzero);
    else if (n16 <= 64 * 16)
        hipLaunchKernelGGL((xprep_wave_kernel<16, SLOTS>), wgrid, block, 0, stream, a, rows, witems,
                           zero, nzero);
    else if (n16 <= 64 * 32)
        hipLaunchKernelGGL((xprep_wave_kernel<32, SLOTS>), wgrid, block, 0, stream, a, rows, witems,
                           zero, nzero);
    else
        hipLaunchKernelGGL((xprep_row_kernel<SLOTS>),
                           dim3((unsigned)std::max<int64_t>(rows, (witems + 31) / 32)), block, 0,
                           stream, a, rows, witems, zero, nzero);
}

}  // namespace

hipError_t launch_xprep(const XprepJob *jobs, int n, const WshiftJob *wjobs, int nw,
                        bool q4_slots, int *zero, int nzero, hipStream_t stream)
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
    int64_t items = 0;
    for (int i = 0; i < nw; ++i) {
        a.w[i] = wjobs[i];
        a.wrow_begin[i] = (int)items;
        items += (int64_t)wjobs[i].parts * wjobs[i].ld;
    }
    a.nw = nw;
    if ((int64_t)rows + items + 32 >= ((int64_t)1 << 31))
        return hipErrorInvalidValue;
    if (q4_slots)
        launch_xprep_t<true>(a, rows, (int)items, maxK, zero, nzero, stream);
    else
        launch_xprep_t<false>(a, rows, (int)items, maxK, zero, nzero, stream);
    return hipGetLastError();
}

}  // namespace qlk
