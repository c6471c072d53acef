// Quantized linear forward for one to four activation rows (bf16): a
// wavefront-reduction GEMV, bound by HBM bandwidth.
//
//   Y[m][n] = sum_b s[n][b] * sum_{k in b} X[m][k] * c[n][k]
//
// Decomposition.  Each wavefront owns RPW weight rows; lane l takes the
// 32-wide blocks l, l + 64, ... of each of them (one block = 32 int8 codes =
// 32 bytes, or 32 q4 codes = 16 bytes, plus one fp16 scale).  All of a
// lane's codes and scales are loaded into registers at the start, before
// anything else, so that every byte the wavefront needs is in flight at once
// (the kernel's runtime is the HBM transfer plus a short tail).  The
// workgroup's four wavefronts share the activations, which are staged once
// per workgroup into LDS while the weight loads are in flight.
//
// Arithmetic (per block, in fp32): per block and activation row, the 32
// products x * c (bf16 x and integer c, exact) are summed in fp32 by bf16
// pair dot products and the block's fp16 scale is applied to that partial
// with one fp32 FMA; the lane partials are then summed across the wavefront
// by DPP steps in a fixed order (deterministic).
//
// Grouping.  One launch takes up to QL_MAX_GROUP layers of one format and
// one row count (a DiT block's four linears): layer i owns the workgroups
// begin[i] .. begin[i + 1] - 1 (the host lists the longest rows first).  The
// blocks per lane (a template bound) are those of the longest K.  A layer
// whose rows fit one block per lane runs a one-block body with twice the
// rows per wavefront instead; a layer in between still issues every load of
// the bound, so that they all go out at once: its lanes past the row's end
// load the row's last block (one line per wavefront) and skip it.
//
// Requirements (checked by the host): M <= 4, K % 256 == 0, M * K <= 32768
// (the activation stage fits LDS), 16-byte aligned codes and X.
#include <algorithm>

#include "epilogue.h"
#include "internal.h"

namespace qlk {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int WAVES = 4;
constexpr int XMAX = 32768;  // activation elements staged per workgroup (64 KB at most)

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

template <int FMT>
struct Block {
    uint32_t w[FMT == QL_FMT_INT8 ? 8 : 4];  // the lane's 32 codes of one block
};

__device__ inline float dot2(uint32_t a, uint32_t b, float c)
{
    return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, a),
                                           __builtin_bit_cast(bf16x2, b), c, false);
}

// high halves of two fp32 -> one bf16 pair (exact for the integer codes)
__device__ inline uint32_t pack_hi(float lo, float hi)
{
    return __builtin_amdgcn_perm(__float_as_uint(hi), __float_as_uint(lo), 0x07060302u);
}

// sum over the block's 32 k of x[k] * w[k] with the activation slice xs (32
// bf16 in LDS), by bf16 pair dot products accumulated in fp32.  int8: w is
// the code itself (sign-extended, converted, packed: exact).  q4: w is the
// offset form 136 + c (bf16 pattern 0x4300 | (nibble ^ 8) = 128 + (c + 8),
// exact), so the result is sum x c + 136 sum x; the caller removes the second
// term.
template <int FMT>
__device__ inline float block_dot(const Block<FMT> &bk, const uint16_t *xs)
{
    float s0 = 0.f, s1 = 0.f;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const u32x4 x = *reinterpret_cast<const u32x4 *>(xs + 8 * q);  // k = 8q .. 8q + 7
        uint32_t w[4];
        if constexpr (FMT == QL_FMT_INT8) {
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                const uint32_t v = bk.w[2 * q + h];
                const float c0 = (float)(int)(int8_t)v, c1 = (float)(int)(int8_t)(v >> 8);
                const float c2 = (float)(int)(int8_t)(v >> 16), c3 = (float)(int)(int8_t)(v >> 24);
                w[2 * h] = pack_hi(c0, c1);
                w[2 * h + 1] = pack_hi(c2, c3);
            }
        } else {
            const uint32_t v = bk.w[q] ^ 0x88888888u, y = v >> 4;
            w[0] = (__builtin_amdgcn_perm(y, v, 0x0C040C00u) & 0x000F000Fu) | 0x43004300u;
            w[1] = (__builtin_amdgcn_perm(y, v, 0x0C050C01u) & 0x000F000Fu) | 0x43004300u;
            w[2] = (__builtin_amdgcn_perm(y, v, 0x0C060C02u) & 0x000F000Fu) | 0x43004300u;
            w[3] = (__builtin_amdgcn_perm(y, v, 0x0C070C03u) & 0x000F000Fu) | 0x43004300u;
        }
        s0 = dot2(x[0], w[0], s0);
        s1 = dot2(x[1], w[1], s1);
        s0 = dot2(x[2], w[2], s0);
        s1 = dot2(x[3], w[3], s1);
    }
    return s0 + s1;
}

// v + (v of another lane), the other lane chosen by the DPP control
template <int CTRL, int ROW_MASK = 0xF>
__device__ inline float dpp_add(float v)
{
    return v + __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(
                                             0, __builtin_bit_cast(int, v), CTRL, ROW_MASK, 0xF,
                                             false));
}

// sum over the 64 lanes: pairs and quads (quad_perm), 8 and 16 lanes (half
// mirror, mirror), then rows carried into rows 1 and 3 and into rows 2 and 3
// (row_bcast 15 / 31); lane 63 ends with the total
__device__ inline float wave_sum(float v)
{
    v = dpp_add<0xB1>(v);        // quad_perm [1, 0, 3, 2]
    v = dpp_add<0x4E>(v);        // quad_perm [2, 3, 0, 1]
    v = dpp_add<0x141>(v);       // row_half_mirror
    v = dpp_add<0x140>(v);       // row_mirror
    v = dpp_add<0x142, 0xA>(v);  // row_bcast:15
    v = dpp_add<0x143, 0xC>(v);  // row_bcast:31
    return v;
}

// The kernel body for workgroup wg of layer d (see the single-layer and
// grouped kernels below)
template <int FMT, int MM, int RPW, int BPL>
__device__ __forceinline__ void gemv_body(const LinDesc &d, const int wg)
{
    // dynamic LDS, sized at launch (M K bf16, then q4's M K / 32 fp32 block
    // sums, for the group's largest K) so that small activations leave room
    // for many workgroups per CU
    extern __shared__ __align__(16) uint16_t xs[];
    float *const xsum = reinterpret_cast<float *>(xs + d.M * d.K);
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int N = d.N, K = d.K, nb = K >> 5;
    const int n0 = (wg * WAVES + wave) * RPW;
    constexpr int CB = FMT == QL_FMT_INT8 ? 32 : 16;  // code bytes per block
    const int crow = FMT == QL_FMT_INT8 ? K : K / 2;

    // 1. the activations' share of this thread, issued first: the stage
    // below then waits only for these, not for the weight loads behind them
    // (loads complete in order)
    const uint16_t *X = reinterpret_cast<const uint16_t *>(d.X);
    const int xe = d.M * K;
    constexpr int XL = MM * BPL;  // K <= 2048 BPL: M K / (8 * 256) loads at most
    u32x4 xv[XL];
#pragma unroll
    for (int j = 0; j < XL; ++j) {
        const int i = (tid + j * 64 * WAVES) * 8;
        if (i < xe)
            xv[j] = *reinterpret_cast<const u32x4 *>(X + i);
    }

    // 2. every code and scale of this lane, in flight before any use
    Block<FMT> bk[RPW][BPL];
    uint16_t sc[RPW][BPL];
#pragma unroll
    for (int r = 0; r < RPW; ++r) {
        const int n = min(n0 + r, N - 1);
        const u32x4 *cr = reinterpret_cast<const u32x4 *>(d.codes + (int64_t)n * crow);
#pragma unroll
        for (int t = 0; t < BPL; ++t) {
            const int b = min(lane + 64 * t, nb - 1);
#pragma unroll
            for (int h = 0; h < CB / 16; ++h) {
                const u32x4 v = __builtin_nontemporal_load(cr + b * (CB / 16) + h);
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    bk[r][t].w[4 * h + e] = v[e];
            }
            sc[r][t] = d.scales[(int64_t)n * nb + b];
        }
    }

    // 3. the activations into LDS, once per workgroup (q4: also 136 * each
    // block's sum of x, fp32)
#pragma unroll
    for (int j = 0; j < XL; ++j) {
        const int i = (tid + j * 64 * WAVES) * 8;
        if (i < xe)
            *reinterpret_cast<u32x4 *>(xs + i) = xv[j];
    }
    __syncthreads();
    if constexpr (FMT == QL_FMT_Q4) {
        for (int i = tid; i < d.M * nb; i += 64 * WAVES) {
            const uint16_t *xb = xs + i * 32;
            float t0 = 0.f, t1 = 0.f;
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const u32x4 x = *reinterpret_cast<const u32x4 *>(xb + 8 * q);
                t0 = dot2(x[0], 0x3F803F80u, t0);  // times bf16 (1, 1)
                t1 = dot2(x[1], 0x3F803F80u, t1);
                t0 = dot2(x[2], 0x3F803F80u, t0);
                t1 = dot2(x[3], 0x3F803F80u, t1);
            }
            xsum[i] = 136.f * (t0 + t1);
        }
        __syncthreads();
    }

    // 4. per block: exact fp32 partial, times the block's scale
    float acc[RPW][MM];
#pragma unroll
    for (int r = 0; r < RPW; ++r)
#pragma unroll
        for (int m = 0; m < MM; ++m)
            acc[r][m] = 0.f;
#pragma unroll
    for (int t = 0; t < BPL; ++t) {
        const int b = lane + 64 * t;
        if (b >= nb)
            continue;
#pragma unroll
        for (int m = 0; m < MM; ++m) {
            const uint16_t *xm = xs + m * K + b * 32;
#pragma unroll
            for (int r = 0; r < RPW; ++r) {
                const float s = (float)__builtin_bit_cast(_Float16, sc[r][t]);
                float p = block_dot<FMT>(bk[r][t], xm);
                if constexpr (FMT == QL_FMT_Q4)
                    p -= xsum[m * nb + b];
                acc[r][m] = __builtin_fmaf(s, p, acc[r][m]);
            }
        }
    }

    // 5. sum over the wavefront in a fixed order (DPP, in registers); lane
    // 63 holds the total and stores
#pragma unroll
    for (int r = 0; r < RPW; ++r)
#pragma unroll
        for (int m = 0; m < MM; ++m)
            acc[r][m] = wave_sum(acc[r][m]);
    if (lane == 63)
#pragma unroll
        for (int r = 0; r < RPW; ++r)
            if (n0 + r < N)
#pragma unroll
                for (int m = 0; m < MM; ++m)
                    epi_store(d.ep, d.Y, (int64_t)m * N + n0 + r, n0 + r, acc[r][m]);
}

template <int FMT, int MM, int RPW, int BPL>
__global__ __launch_bounds__(64 * WAVES) void qgemv_kernel(const LinDesc d)
{
    gemv_body<FMT, MM, RPW, BPL>(d, (int)blockIdx.x);
}

// rows per wavefront for a layer of the group: a layer whose rows fit one
// block per lane takes twice the group's rows per wavefront (the same
// registers as the longer layers' blocks, and half the workgroups)
template <int RPW, int BPL>
__host__ __device__ inline int group_rpw(int K)
{
    return BPL > 1 && K / 32 <= 64 ? 2 * RPW : RPW;
}

template <int FMT, int MM, int RPW, int BPL>
__global__ __launch_bounds__(64 * WAVES) void qgemv_group_kernel(const LayerGroup grp)
{
    // this workgroup's layer (wave-uniform) and its index within the layer;
    // a layer of one block per lane runs the one-block body (its loads and
    // registers only)
    int li = 0;
    while (li + 1 < grp.n && (int)blockIdx.x >= grp.begin[li + 1])
        ++li;
    const int wg = (int)blockIdx.x - grp.begin[li];
    if (group_rpw<RPW, BPL>(grp.d[li].K) != RPW)
        gemv_body<FMT, MM, 2 * RPW, 1>(grp.d[li], wg);
    else
        gemv_body<FMT, MM, RPW, BPL>(grp.d[li], wg);
}

template <int FMT, int MM, int RPW, int BPL>
void launch_one(const LayerGroup &g, dim3 grid, size_t lds, hipStream_t s)
{
    if (g.n == 1)
        hipLaunchKernelGGL((qgemv_kernel<FMT, MM, RPW, BPL>), grid, dim3(64 * WAVES), lds, s,
                           g.d[0]);
    else
        hipLaunchKernelGGL((qgemv_group_kernel<FMT, MM, RPW, BPL>), grid, dim3(64 * WAVES), lds,
                           s, g);
}

template <int FMT, int MM, int RPW>
hipError_t launch_bpl(const LayerGroup &g0, hipStream_t s)
{
    LayerGroup g = g0;
    int nbmax = 0;
    size_t lds = 0;
    for (int i = 0; i < g.n; ++i) {
        const LinDesc &d = g.d[i];
        const int nb = d.K / 32;
        nbmax = std::max(nbmax, nb);
        lds = std::max(lds, (size_t)d.M * d.K * 2 +
                                (FMT == QL_FMT_Q4 ? (size_t)d.M * nb * 4 : 0));
    }
    const int bpl = (nbmax + 63) / 64;
    // workgroups per layer: rows per wavefront as the group kernel takes them
    g.begin[0] = 0;
    for (int i = 0; i < g.n; ++i) {
        const int rpw = g.n > 1 && bpl > 1 && g.d[i].K / 32 <= 64 ? 2 * RPW : RPW;
        g.begin[i + 1] = g.begin[i] + (g.d[i].N + WAVES * rpw - 1) / (WAVES * rpw);
    }
    const dim3 grid((unsigned)g.begin[g.n]);
    switch (bpl) {
    case 1: launch_one<FMT, MM, RPW, 1>(g, grid, lds, s); break;
    case 2: launch_one<FMT, MM, RPW, 2>(g, grid, lds, s); break;
    case 3: launch_one<FMT, MM, RPW, 3>(g, grid, lds, s); break;
    case 4: launch_one<FMT, MM, RPW, 4>(g, grid, lds, s); break;
    default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

template <int FMT>
hipError_t launch_fmt(const LayerGroup &g, hipStream_t s)
{
    // two weight rows per wavefront while that still leaves two workgroups
    // per CU, one otherwise; q4 at two activation rows keeps one (a d = 2048
    // block 14.6 -> 13.0 us; int8 at two rows and both formats at three and
    // four measured slower with one)
    int64_t rows = 0;
    for (int i = 0; i < g.n; ++i)
        rows += g.d[i].N;
    const bool two = !(FMT == QL_FMT_Q4 && g.d[0].M == 2) &&
                     (rows + 2 * WAVES - 1) / (2 * WAVES) >= 512;
    switch (g.d[0].M) {
    case 1: return two ? launch_bpl<FMT, 1, 2>(g, s) : launch_bpl<FMT, 1, 1>(g, s);
    case 2: return two ? launch_bpl<FMT, 2, 2>(g, s) : launch_bpl<FMT, 2, 1>(g, s);
    case 3: return two ? launch_bpl<FMT, 3, 2>(g, s) : launch_bpl<FMT, 3, 1>(g, s);
    case 4: return two ? launch_bpl<FMT, 4, 2>(g, s) : launch_bpl<FMT, 4, 1>(g, s);
    default: return hipErrorInvalidValue;
    }
}

}  // namespace

bool gemv_ok(const LinDesc &d)
{
    return d.M >= 1 && d.M <= 4 && d.K % 256 == 0 && d.K <= 8192 && (int64_t)d.M * d.K <= XMAX;
}

hipError_t launch_qgemv(int fmt, const LayerGroup &g, hipStream_t stream)
{
    for (int i = 1; i < g.n; ++i)
        if (g.d[i].M != g.d[0].M)
            return hipErrorInvalidValue;  // one row count per launch
    return fmt == QL_FMT_INT8 ? launch_fmt<QL_FMT_INT8>(g, stream)
                              : launch_fmt<QL_FMT_Q4>(g, stream);
}

}  // namespace qlk
