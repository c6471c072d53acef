// Quantized linear forward on the MI355X matrix cores.
//
//   Y[m][n] = sum_b s[n][b] * sum_{k in b} X[m][k] * c[n][k]
//
// (paper: Methodology, "Quantization and its evaluation" — the linears run
// from the 8-bit / 4-bit weight copy; block of 32 along K, fp16 scale).
//
// Numerics.  Each 32-wide K block is one v_mfma_f32_16x16x32_bf16, so the
// block partial sum is formed from the *exact* integer codes (every code and
// code + offset below is an integer < 2^8, exact in bf16) and the bf16
// activations, with fp32 accumulation; the fp16 scale is then applied in fp32
// (acc += s * partial).  Folding the scale into a bf16 weight instead would
// round every weight to 8 significant bits.  fp32 activations are split
// exactly into three bf16 terms (hi + mid + lo == x) and contracted with
// three chained MFMAs, so fp32 inputs keep fp32 accuracy.
//
// Cheap code -> bf16 conversion (bf16 activations only).  Codes are fed to
// the MFMA with a constant offset so that no sign handling is needed:
//   int8: byte ^ 0x80 = c + 128 in [0, 255], converted by v_cvt_f32_ubyteN
//   q4:   nibble ^ 8 = c + 8, OR-ed into the bf16 pattern 0x4300 (= 128), so
//         two codes become one packed bf16 pair (136 + c) with one AND-OR.
// The offset's contribution OFF * sum_{k in b} X[m][k] depends only on
// (m, b); it is computed once per tile row while staging X and enters the
// MFMA through its C operand as -OFF * sum, so the partial that leaves the
// MFMA is already offset-free.  The q4 trick pairs codes (k, k+4) in one
// register, so the staged activations are permuted the same way.
//
// Tiling.  256 threads = 4 wavefronts per workgroup; a workgroup computes a
// BM x BN tile of Y (BM = 16*MSUB rows of X, BN = 4 * 16*NSUB rows of W);
// each wavefront owns NSUB 16-wide column strips and all BM rows, so every
// code is loaded and converted exactly once per workgroup and reused for all
// MSUB row subtiles.  X is staged through LDS two K blocks (64 k) at a time,
// double-buffered, with one barrier per step; codes and scales stream from
// HBM straight into registers one step ahead.  Workgroups are assigned to
// tiles XCD-aware: the 8 XCDs take contiguous ranges of the logical tile
// order (row tiles fastest), so workgroups sharing a weight strip share an
// L2.  A long reduction with too few tiles for the GPU is cut into K parts
// (LinDesc::ksplit parts of psteps 64-k steps): each part stores a plain
// fp32 partial output and the split-sum launch adds them in part order.
#include <type_traits>

#include "epilogue.h"
#include "internal.h"

namespace qlk {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int RS = 40;  // LDS row stride in bf16 elements: 32 + 8 pad (80 B)

__device__ inline f32x4 mfma(u32x4 a, u32x4 b, f32x4 c)
{
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                   __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

__device__ inline uint32_t pack_hi16(float lo, float hi)
{
    // both values are small integers: the bf16 pattern is the fp32 high half
    return (__float_as_uint(lo) >> 16) | (__float_as_uint(hi) & 0xFFFF0000u);
}

__device__ inline float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ inline float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

// ---- code conversion ------------------------------------------------------
// int8, offset form: 8 codes (k0..k7) -> bf16 of c + 128, natural k order.
__device__ inline u32x4 cvt_int8_off(uint2 c)
{
    const uint32_t a = c.x ^ 0x80808080u, b = c.y ^ 0x80808080u;
    u32x4 r;
    r[0] = pack_hi16((float)(a & 0xFF), (float)((a >> 8) & 0xFF));
    r[1] = pack_hi16((float)((a >> 16) & 0xFF), (float)(a >> 24));
    r[2] = pack_hi16((float)(b & 0xFF), (float)((b >> 8) & 0xFF));
    r[3] = pack_hi16((float)((b >> 16) & 0xFF), (float)(b >> 24));
    return r;
}

// q4, offset form: 8 codes (one dword, k0 in bits 0-3) -> bf16 of c + 136 in
// the order (k0,k4), (k1,k5), (k2,k6), (k3,k7).
__device__ inline u32x4 cvt_q4_off(uint32_t c)
{
    const uint32_t x = c ^ 0x88888888u;
    u32x4 r;
    r[0] = (x & 0x000F000Fu) | 0x43004300u;
    r[1] = ((x >> 4) & 0x000F000Fu) | 0x43004300u;
    r[2] = ((x >> 8) & 0x000F000Fu) | 0x43004300u;
    r[3] = ((x >> 12) & 0x000F000Fu) | 0x43004300u;
    return r;
}

// int8, exact signed form, natural k order.
__device__ inline u32x4 cvt_int8_exact(uint2 c)
{
    u32x4 r;
    r[0] = pack_hi16((float)(int8_t)(c.x & 0xFF), (float)(int8_t)((c.x >> 8) & 0xFF));
    r[1] = pack_hi16((float)(int8_t)((c.x >> 16) & 0xFF), (float)(int8_t)(c.x >> 24));
    r[2] = pack_hi16((float)(int8_t)(c.y & 0xFF), (float)(int8_t)((c.y >> 8) & 0xFF));
    r[3] = pack_hi16((float)(int8_t)((c.y >> 16) & 0xFF), (float)(int8_t)(c.y >> 24));
    return r;
}

// q4, exact signed form, natural k order.
__device__ inline u32x4 cvt_q4_exact(uint32_t c)
{
    float f[8];
#pragma unroll
    for (int j = 0; j < 8; ++j)
        f[j] = (float)(((int32_t)(c << (28 - 4 * j))) >> 28);
    u32x4 r;
    r[0] = pack_hi16(f[0], f[1]);
    r[1] = pack_hi16(f[2], f[3]);
    r[2] = pack_hi16(f[4], f[5]);
    r[3] = pack_hi16(f[6], f[7]);
    return r;
}

// (x0..x7) -> (x0,x4), (x1,x5), (x2,x6), (x3,x7), matching cvt_q4_off.
__device__ inline u32x4 permute_q4(u32x4 v)
{
    u32x4 r;
    r[0] = (v[0] & 0xFFFFu) | (v[2] << 16);
    r[1] = (v[0] >> 16) | (v[2] & 0xFFFF0000u);
    r[2] = (v[1] & 0xFFFFu) | (v[3] << 16);
    r[3] = (v[1] >> 16) | (v[3] & 0xFFFF0000u);
    return r;
}

__device__ inline float sum8_bf16(u32x4 v)
{
    float s = 0.f;
#pragma unroll
    for (int j = 0; j < 4; ++j)
        s += bf16_lo(v[j]) + bf16_hi(v[j]);
    return s;
}

// Exact split of 8 fp32 values into bf16 hi / mid / lo planes.
__device__ inline void split3(const u32x4 &p0, const u32x4 &p1, u32x4 &hi, u32x4 &mid,
                              u32x4 &lo)
{
    uint32_t h[8], m[8], l[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        const uint32_t xb = j < 4 ? p0[j] : p1[j - 4];
        const float x = __uint_as_float(xb);
        const uint32_t hb = xb & 0xFFFF0000u;
        const float r1 = x - __uint_as_float(hb);
        const uint32_t mb = __float_as_uint(r1) & 0xFFFF0000u;
        const float r2 = r1 - __uint_as_float(mb);
        h[j] = hb >> 16;
        m[j] = mb >> 16;
        l[j] = __float_as_uint(r2) >> 16;
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        hi[j] = h[2 * j] | (h[2 * j + 1] << 16);
        mid[j] = m[2 * j] | (m[2 * j + 1] << 16);
        lo[j] = l[2 * j] | (l[2 * j + 1] << 16);
    }
}

__device__ inline int logical_tile(int p, int G)
{
    // hardware places workgroup p on XCD p % 8; give each XCD a contiguous
    // range of logical tiles (XCDs 0..r-1 take q+1 tiles, the rest q).
    const int q = G >> 3, r = G & 7;
    const int xcd = p & 7, idx = p >> 3;
    return xcd < r ? xcd * (q + 1) + idx : r * (q + 1) + (xcd - r) * q + idx;
}

template <int FMT, bool XF32, int MSUB, int NSUB>
__global__ __launch_bounds__(256) void qgemm_kernel(const GroupArgs args)
{
    constexpr int BM = 16 * MSUB;
    constexpr int NPL = XF32 ? 3 : 1;                   // bf16 planes of X
    constexpr int OFF = FMT == QL_FMT_INT8 ? 128 : 136; // code offset (bf16 X only)
    constexpr int CHUNKS = BM * 8;                      // 8-element chunks per 64-k step
    constexpr int CPT = (CHUNKS + 255) / 256;           // chunks per thread

    __shared__ __align__(16) uint16_t xs[2][NPL][2][BM * RS];
    __shared__ __align__(16) float ts[2][2][XF32 ? 1 : BM];

    // ---- tile of this workgroup ------------------------------------------
    // workgroup p belongs to the layer whose tile range holds p, so every
    // layer (long reductions first) is spread over all 8 XCDs; within the
    // layer, each XCD takes a contiguous range of its tiles
    const int p = (int)blockIdx.x;
    LinDesc d = args.d[0];
    int end = args.total_tiles;
#pragma unroll
    for (int t = 1; t < QL_MAX_GROUP; ++t) {
        if (t < args.n && p >= args.d[t].tile_begin)
            d = args.d[t];
        if (t < args.n && p < args.d[t].tile_begin && end == args.total_tiles)
            end = args.d[t].tile_begin;
    }
    // a split layer's logical tiles walk its K parts fastest
    const int local = logical_tile(p - d.tile_begin, end - d.tile_begin);
    const int S = d.ksplit, part = local % S;
    const int tile = local / S;
    const int tm = tile % d.tiles_m;
    const int tn = tile / d.tiles_m;
    const int M = d.M, N = d.N, K = d.K;
    const int nb = K >> 5;
    const int m0 = tm * BM;

    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int l16 = lane & 15, lg = lane >> 4;
    const int n_wave = tn * (64 * NSUB) + wave * (16 * NSUB);

    // ---- per-lane weight rows ----------------------------------------------
    const uint8_t *crow[NSUB];
    const uint16_t *srow[NSUB];
#pragma unroll
    for (int j = 0; j < NSUB; ++j) {
        int n = n_wave + j * 16 + l16;
        n = n < N ? n : N - 1;
        crow[j] = d.codes + (int64_t)n * (FMT == QL_FMT_INT8 ? K : K / 2) +
                  (FMT == QL_FMT_INT8 ? lg * 8 : lg * 4);
        srow[j] = d.scales + (int64_t)n * nb;
    }

    // ---- staging of X (global -> registers -> LDS) -------------------------
    u32x4 xr[CPT][XF32 ? 2 : 1];
    auto load_x = [&](int step) {
#pragma unroll
        for (int q = 0; q < CPT; ++q) {
            const int c = tid + 256 * q;
            const int row = c >> 3, part = c & 7;
            const int kb = 2 * step + (part >> 2);
            const int m = m0 + row;
            const bool ok = c < CHUNKS && m < M && kb < nb;
            const int64_t off = (int64_t)m * K + kb * 32 + (part & 3) * 8;
#pragma unroll
            for (int h = 0; h < (XF32 ? 2 : 1); ++h) {
                u32x4 v = {0u, 0u, 0u, 0u};
                if (ok) {
                    if (XF32)
                        v = *reinterpret_cast<const u32x4 *>(
                            reinterpret_cast<const float *>(d.X) + off + 4 * h);
                    else
                        v = *reinterpret_cast<const u32x4 *>(
                            reinterpret_cast<const uint16_t *>(d.X) + off);
                }
                xr[q][h] = v;
            }
        }
    };
    auto store_x = [&](int buf) {
#pragma unroll
        for (int q = 0; q < CPT; ++q) {
            const int c = tid + 256 * q;
            const int row = c >> 3, part = c & 7;
            const int blk = part >> 2, g = part & 3;
            if (XF32) {
                u32x4 hi, mid, lo;
                split3(xr[q][0], xr[q][1], hi, mid, lo);
                if (c < CHUNKS) {
                    *reinterpret_cast<u32x4 *>(&xs[buf][0][blk][row * RS + g * 8]) = hi;
                    *reinterpret_cast<u32x4 *>(&xs[buf][NPL > 1 ? 1 : 0][blk][row * RS + g * 8]) = mid;
                    *reinterpret_cast<u32x4 *>(&xs[buf][NPL > 2 ? 2 : 0][blk][row * RS + g * 8]) = lo;
                }
            } else {
                const u32x4 v = xr[q][0];
                float s = sum8_bf16(v);
                s += __shfl_xor(s, 1);
                s += __shfl_xor(s, 2);
                if (c < CHUNKS) {
                    *reinterpret_cast<u32x4 *>(&xs[buf][0][blk][row * RS + g * 8]) =
                        FMT == QL_FMT_Q4 ? permute_q4(v) : v;
                    if (g == 0)
                        ts[buf][blk][XF32 ? 0 : row] = -(float)OFF * s;
                }
            }
        }
    };

    // ---- codes and scales (global -> registers, one step ahead) -----------
    typedef typename std::conditional<FMT == QL_FMT_INT8, uint2, uint32_t>::type CodeT;
    CodeT cr[2][NSUB], cn[2][NSUB];
    uint16_t sr[2][NSUB], sn[2][NSUB];
    auto load_codes = [&](int step, CodeT (&c)[2][NSUB], uint16_t (&s)[2][NSUB]) {
#pragma unroll
        for (int bi = 0; bi < 2; ++bi) {
            const int kb = 2 * step + bi;
            if (kb < nb) {
#pragma unroll
                for (int j = 0; j < NSUB; ++j) {
                    c[bi][j] = *reinterpret_cast<const CodeT *>(
                        crow[j] + (int64_t)kb * (FMT == QL_FMT_INT8 ? 32 : 16));
                    s[bi][j] = srow[j][kb];
                }
            }
        }
    };

    f32x4 acc[MSUB][NSUB];
#pragma unroll
    for (int i = 0; i < MSUB; ++i)
#pragma unroll
        for (int j = 0; j < NSUB; ++j)
            acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    // this part's 64-k steps [s0, s1)
    const int s0 = part * d.psteps;
    const int s1 = min((nb + 1) >> 1, s0 + d.psteps);
    load_codes(s0, cr, sr);
    load_x(s0);
    store_x(0);
    __syncthreads();

    for (int step = s0; step < s1; ++step) {
        const int buf = (step - s0) & 1;
        const bool more = step + 1 < s1;
        if (more) {
            load_x(step + 1);
            load_codes(step + 1, cn, sn);
        }
        const int nblk = nb - 2 * step < 2 ? 1 : 2;
#pragma unroll
        for (int bi = 0; bi < 2; ++bi) {
            if (bi < nblk) {
                u32x4 B[NSUB];
                float sc[NSUB];
#pragma unroll
                for (int j = 0; j < NSUB; ++j) {
                    if (XF32)
                        B[j] = FMT == QL_FMT_INT8 ? cvt_int8_exact(*(uint2 *)&cr[bi][j])
                                                  : cvt_q4_exact(*(uint32_t *)&cr[bi][j]);
                    else
                        B[j] = FMT == QL_FMT_INT8 ? cvt_int8_off(*(uint2 *)&cr[bi][j])
                                                  : cvt_q4_off(*(uint32_t *)&cr[bi][j]);
                    sc[j] = (float)__builtin_bit_cast(_Float16, sr[bi][j]);
                }
                // all MFMAs of this block first (independent partials), then
                // the per-block scale, so MFMA latency overlaps the FMAs
                f32x4 P[MSUB][NSUB];
#pragma unroll
                for (int i = 0; i < MSUB; ++i) {
                    const int ro = (i * 16 + l16) * RS + lg * 8;
                    const u32x4 a0 = *reinterpret_cast<const u32x4 *>(&xs[buf][0][bi][ro]);
                    f32x4 cin = {0.f, 0.f, 0.f, 0.f};
                    if (!XF32)
                        cin = *reinterpret_cast<const f32x4 *>(&ts[buf][bi][XF32 ? 0 : i * 16 + lg * 4]);
                    u32x4 a1 = a0, a2 = a0;
                    if (XF32) {
                        a1 = *reinterpret_cast<const u32x4 *>(&xs[buf][NPL > 1 ? 1 : 0][bi][ro]);
                        a2 = *reinterpret_cast<const u32x4 *>(&xs[buf][NPL > 2 ? 2 : 0][bi][ro]);
                    }
#pragma unroll
                    for (int j = 0; j < NSUB; ++j) {
                        f32x4 p = mfma(a0, B[j], cin);
                        if (XF32) {
                            p = mfma(a1, B[j], p);
                            p = mfma(a2, B[j], p);
                        }
                        P[i][j] = p;
                    }
                }
#pragma unroll
                for (int i = 0; i < MSUB; ++i)
#pragma unroll
                    for (int j = 0; j < NSUB; ++j)
                        acc[i][j] += sc[j] * P[i][j];
            }
        }
        if (more) {
            store_x(buf ^ 1);
#pragma unroll
            for (int bi = 0; bi < 2; ++bi)
#pragma unroll
                for (int j = 0; j < NSUB; ++j) {
                    cr[bi][j] = cn[bi][j];
                    sr[bi][j] = sn[bi][j];
                }
        }
        __syncthreads();
    }

    // ---- epilogue: lane holds rows 4*lg + r of each 16-row subtile; a part
    // of a split layer stores its plain partial output (the sum launch adds
    // the parts and applies the epilogue) --------------------------------
    float *const Yp = S > 1 ? d.part + (int64_t)part * M * N : nullptr;
#pragma unroll
    for (int i = 0; i < MSUB; ++i)
#pragma unroll
        for (int j = 0; j < NSUB; ++j) {
            const int n = n_wave + j * 16 + l16;
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int m = m0 + i * 16 + lg * 4 + r;
                if (m < M && n < N) {
                    if (S > 1)
                        Yp[(int64_t)m * N + n] = acc[i][j][r];
                    else
                        epi_store(d.ep, d.Y, (int64_t)m * N + n, n, acc[i][j][r]);
                }
            }
        }
}

template <int FMT, bool XF32>
hipError_t launch_fx(TileCfg t, const GroupArgs &a, hipStream_t s)
{
    dim3 grid((unsigned)a.total_tiles), block(256);
    switch (t) {
    case TILE_M16:
        hipLaunchKernelGGL((qgemm_kernel<FMT, XF32, 1, 1>), grid, block, 0, s, a);
        break;
    case TILE_M32:
        hipLaunchKernelGGL((qgemm_kernel<FMT, XF32, 2, 1>), grid, block, 0, s, a);
        break;
    case TILE_M64:
        hipLaunchKernelGGL((qgemm_kernel<FMT, XF32, 4, 2>), grid, block, 0, s, a);
        break;
    default:
        // fp32 activations use three LDS planes: the 128-row tile is not built
        if (XF32)
            return hipErrorInvalidValue;
        hipLaunchKernelGGL((qgemm_kernel<FMT, false, 8, 2>), grid, block, 0, s, a);
        break;
    }
    return hipGetLastError();
}

}  // namespace

int tile_bm(TileCfg t)
{
    return t == TILE_M16 ? 16 : t == TILE_M32 ? 32 : t == TILE_M64 ? 64 : 128;
}

int tile_bn(TileCfg t)
{
    return t == TILE_M16 || t == TILE_M32 ? 64 : 128;
}

hipError_t launch_qgemm(int fmt, bool xf32, TileCfg t, const GroupArgs &args,
                        hipStream_t stream)
{
    if (fmt == QL_FMT_INT8)
        return xf32 ? launch_fx<QL_FMT_INT8, true>(t, args, stream)
                    : launch_fx<QL_FMT_INT8, false>(t, args, stream);
    return xf32 ? launch_fx<QL_FMT_Q4, true>(t, args, stream)
                : launch_fx<QL_FMT_Q4, false>(t, args, stream);
}

}  // namespace qlk
