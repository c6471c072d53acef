// Quantized linear forward, large-M tile (bf16 activations, M > 64,
// K a multiple of 64, 4-byte aligned scales).
//
//   Y[m][n] = sum_b s[n][b] * sum_{k in b} X[m][k] * c[n][k]
//
// Numerics: one v_mfma_f32_16x16x32_bf16 per 32-wide K block contracts the
// bf16 activations with integer codes that are exact in bf16; the fp16 block
// scale is then applied to the fp32 partial with one FMA per output element
// per block.  int8 codes are converted exactly (sign-extending
// v_cvt_f32_i32 on each byte, fp32 high halves packed by v_perm).  q4 codes
// take the cheaper offset form 0x4300 | (nibble ^ 8) = bf16(136 + c), two
// codes per AND-OR; the offset's contribution -136 * sum_{k in b} X[m][k]
// comes from one extra MFMA of the activation fragment against a constant
// -136 matrix and enters each main MFMA as its C operand.  The kernel is
// bound by VALU issue (the per-block scale FMAs cost as much issue time as
// the MFMAs), so trading conversion work for matrix-core work pays.
//
// Tile: 256 threads (4 wavefronts) compute BM x BN = 128 x 128 of Y.  Each
// wavefront owns a 128 x 32 strip (8 x 2 MFMA subtiles), so every converted
// code fragment feeds 8 MFMAs and every activation fragment 2.
//
// Memory pipeline: activations, codes and scales move from HBM to LDS with
// the gfx950 direct-to-LDS loads (no VGPRs, no VALU), through a ring of 3
// stages of 64 k (two scale blocks) each; a stage is issued two steps before
// it is consumed and the main loop is unrolled by the ring depth so each
// stage's LDS slot is fixed.  Each lane's global offset within the tile is
// computed once; per step only the wave-uniform base address (an SGPR pair)
// advances.  The loads are issued from inline asm so that the compiler's wait
// insertion, which cannot tell the ring stages apart and would drain every
// load in flight before each LDS read, stays out of the way: the kernel waits
// for each stage explicitly (s_waitcnt vmcnt + s_barrier; a __syncthreads()
// would also drain the ring).  Nothing else in these kernels uses M0.
//
// LDS layouts are XOR-swizzled at 16-byte granularity so that the fragment
// reads (16 rows x 16 B per 16 lanes) hit distinct banks.  A direct-to-LDS
// load writes lane t's data to slot base + t, so the swizzle is applied by
// choosing which global chunk each lane fetches.
//
// fp16 variant (F16): the host first converts the activations exactly to
// fp16 with a per-row power-of-two shift (xprep.hip); the kernel pre-scans the
// tile's scales for a shift f that keeps every |c * s * 2^-f| <= Q * smax *
// 2^-f < 2^15, dequantizes each weight to fp16 (c exact in fp16 by a
// magic-number add, then one rounded packed multiply by s * 2^-f), and
// accumulates the whole K inside v_mfma_f32_16x16x32_f16, so the per-block
// scale FMAs disappear.  The only rounding beyond fp32 accumulation is that
// of c * s to 11 significant bits (~2e-4 of max|Y| at the DiT shapes,
// against the 2e-3 tolerance).  The epilogue applies both shifts exactly.
//
// Tile order: within a layer, groups of 4 row tiles walked row-tile fastest;
// each of the 8 XCDs takes a contiguous range of one layer's tiles (L2
// reuse), and every layer of a grouped launch is spread over all XCDs.
#include "internal.h"

namespace qlk {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef _Float16 half2v __attribute__((ext_vector_type(2)));

constexpr int MSUB = 8, NSUB = 2, BM = 16 * MSUB, BN = 64 * NSUB, NST = 3, GROUP_M = 4;

template <int FMT>
struct Geo {
    static constexpr int XBYTES = BM * 64 * 2;                 // activations per stage
    static constexpr int CROW = FMT == QL_FMT_INT8 ? 64 : 32;  // code bytes per row per stage
    static constexpr int CBYTES = BN * CROW;
    static constexpr int SBYTES = BN * 4;                      // both scales of a step, per row
    static constexpr int STAGE = XBYTES + CBYTES + SBYTES;
    static constexpr int XLOADS = XBYTES / 16 / 256;
    static constexpr int CLOADS = CBYTES / 16 / 256;
    static constexpr int LOADS = XLOADS + CLOADS + 1;          // direct-to-LDS loads per stage
    static_assert(XBYTES % (16 * 256) == 0 && CBYTES % (16 * 256) == 0,
                  "every thread issues the same number of 16-byte loads per stage");
    static_assert(BN % 64 == 0 && BN <= 256, "one scale dword per weight row per stage");
};

__device__ inline constexpr int vmcnt_imm(int v)
{
    // gfx9 s_waitcnt encoding: vmcnt[3:0] + vmcnt[5:4] at bits 15:14;
    // expcnt (bits 6:4) and lgkmcnt (bits 11:8) left at "no wait"
    return (v & 15) | (((v >> 4) & 3) << 14) | (7 << 4) | (15 << 8);
}

// activation chunk swizzle: the 16 rows one MFMA operand read touches land
// on distinct banks whether the LDS serves 8 lanes of a 16-byte read per
// clock from 32 banks or 16 lanes from 64 banks
__device__ inline int xswz(int row) { return ((row >> 1) & 3) ^ ((row >> 3) & 1); }

// s_waitcnt lgkmcnt(0) with vmcnt and expcnt left at "no wait"
__device__ inline constexpr int lgkm0_imm() { return 15 | (3 << 14) | (7 << 4); }

// Direct-to-LDS loads from (wave-uniform base + per-lane 32-bit offset):
// lane t's data lands at LDS address lds + t * size.
__device__ inline void dma16(const void *base, uint32_t off, uint32_t lds)
{
    asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1"
                 :
                 : "v"(off), "s"(base), "s"(__builtin_amdgcn_readfirstlane(lds))
                 : "memory");
}

__device__ inline void dma4(const void *base, uint32_t off, uint32_t lds)
{
    asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dword %0, %1"
                 :
                 : "v"(off), "s"(base), "s"(__builtin_amdgcn_readfirstlane(lds))
                 : "memory");
}

__device__ inline uint32_t lds_addr(const void *p)
{
    // a generic pointer into LDS carries the LDS offset in its low 32 bits
    return (uint32_t)(uintptr_t)p;
}

__device__ inline f32x4 mfma(u32x4 a, u32x4 b, f32x4 c)
{
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                   __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

__device__ inline f32x4 mfma_f16(u32x4 a, u32x4 b, f32x4 c)
{
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(half8, a),
                                                  __builtin_bit_cast(half8, b), c, 0, 0, 0);
}

__device__ inline uint32_t h2mul_add(uint32_t v, half2v bias, half2v sp)
{
    // (v + bias) exact (an fp16 integer), then one rounded multiply
    return __builtin_bit_cast(uint32_t, (__builtin_bit_cast(half2v, v) + bias) * sp);
}

// 8 int8 codes -> 8 fp16 of c * s', natural order.  byte ^ 0x80 = c + 128 is
// placed under the fp16 pattern 0x64 (= 1024 + (c + 128)) by v_perm; adding
// -1152 leaves c exactly.
__device__ inline u32x4 deq_int8_f16(uint32_t a, uint32_t b, half2v sp)
{
    const uint32_t x = a ^ 0x80808080u, y = b ^ 0x80808080u, hi = 0x64646464u;
    const half2v bias = {(_Float16)-1152.0f, (_Float16)-1152.0f};
    u32x4 r;
    r[0] = h2mul_add(__builtin_amdgcn_perm(hi, x, 0x04010400u), bias, sp);
    r[1] = h2mul_add(__builtin_amdgcn_perm(hi, x, 0x04030402u), bias, sp);
    r[2] = h2mul_add(__builtin_amdgcn_perm(hi, y, 0x04010400u), bias, sp);
    r[3] = h2mul_add(__builtin_amdgcn_perm(hi, y, 0x04030402u), bias, sp);
    return r;
}

// 8 q4 codes -> 8 fp16 of c * s', natural order: nibble ^ 8 = c + 8 under
// the fp16 pattern 0x6400 (= 1024 + c + 8); adding -1032 leaves c exactly.
__device__ inline u32x4 deq_q4_f16(uint32_t c, half2v sp)
{
    const uint32_t x = c ^ 0x88888888u, y = x >> 4;
    const half2v bias = {(_Float16)-1032.0f, (_Float16)-1032.0f};
    u32x4 r;
    r[0] = h2mul_add((__builtin_amdgcn_perm(y, x, 0x0C040C00u) & 0x000F000Fu) | 0x64006400u, bias, sp);
    r[1] = h2mul_add((__builtin_amdgcn_perm(y, x, 0x0C050C01u) & 0x000F000Fu) | 0x64006400u, bias, sp);
    r[2] = h2mul_add((__builtin_amdgcn_perm(y, x, 0x0C060C02u) & 0x000F000Fu) | 0x64006400u, bias, sp);
    r[3] = h2mul_add((__builtin_amdgcn_perm(y, x, 0x0C070C03u) & 0x000F000Fu) | 0x64006400u, bias, sp);
    return r;
}

// fp32 high halves of (lo, hi) as a bf16 pair (exact for small integers)
__device__ inline uint32_t pack_hi(float lo, float hi)
{
    return __builtin_amdgcn_perm(__float_as_uint(hi), __float_as_uint(lo), 0x07060302u);
}

// Signed byte J of x as a float.
template <int J>
__device__ inline float sbyte(uint32_t x)
{
    return (float)((int32_t)(x << (24 - 8 * J)) >> 24);
}

// 8 int8 codes (k0..k7) -> 8 bf16, exact, natural order.
__device__ inline u32x4 cvt_int8(uint32_t a, uint32_t b)
{
    u32x4 r;
    r[0] = pack_hi(sbyte<0>(a), sbyte<1>(a));
    r[1] = pack_hi(sbyte<2>(a), sbyte<3>(a));
    r[2] = pack_hi(sbyte<0>(b), sbyte<1>(b));
    r[3] = pack_hi(sbyte<2>(b), sbyte<3>(b));
    return r;
}

// 8 q4 codes (k0 in bits 0-3) -> bf16 of 136 + c, natural order: byte j of
// x holds codes 2j and 2j+1; v_perm puts byte j of x and of x >> 4 in the two
// 16-bit halves, the AND keeps one nibble in each, the OR adds bf16 128.
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

__device__ inline int logical_tile(int p, int G)
{
    const int q = G >> 3, r = G & 7;
    const int xcd = p & 7, idx = p >> 3;
    return xcd < r ? xcd * (q + 1) + idx : r * (q + 1) + (xcd - r) * q + idx;
}

template <int FMT>
struct Ctx {
    // wave-uniform bases of this tile (advanced per step by the caller)
    const uint8_t *xbase, *cbase, *sbase;
    // per-lane byte offsets from those bases, fixed for the whole K loop
    uint32_t xoff[Geo<FMT>::XLOADS], coff[Geo<FMT>::CLOADS], soff;
    int wave, l16, lg;
    int negf;  // F16: weights enter as c * s * 2^negf
};

// Issue the direct-to-LDS loads of step s into one ring stage.
template <int FMT>
__device__ inline void issue_stage(const Ctx<FMT> &c, uint8_t *stage, int s)
{
    using G = Geo<FMT>;
    const uint32_t base = lds_addr(stage);
    const uint8_t *xb = c.xbase + s * 128;              // 64 bf16 per row per step
    const uint8_t *cb = c.cbase + s * G::CROW;
    const uint8_t *sb = c.sbase + s * 4;
#pragma unroll
    for (int r = 0; r < G::XLOADS; ++r)
        dma16(xb, c.xoff[r], base + (r * 256 + c.wave * 64) * 16);
#pragma unroll
    for (int r = 0; r < G::CLOADS; ++r)
        dma16(cb, c.coff[r], base + G::XBYTES + (r * 256 + c.wave * 64) * 16);
    dma4(sb, c.soff, base + G::XBYTES + G::CBYTES + (c.wave % (BN / 64)) * 256);
}

template <int FMT>
__device__ inline void compute_stage_f16(const Ctx<FMT> &c, const uint8_t *stage,
                                         f32x4 (&acc)[MSUB][NSUB])
{
    using G = Geo<FMT>;
    uint32_t sc[NSUB];
#pragma unroll
    for (int j = 0; j < NSUB; ++j)
        sc[j] = *reinterpret_cast<const uint32_t *>(stage + G::XBYTES + G::CBYTES +
                                                    (c.wave * (16 * NSUB) + j * 16 + c.l16) * 4);
#pragma unroll
    for (int bi = 0; bi < 2; ++bi) {
        u32x4 B[NSUB];
#pragma unroll
        for (int j = 0; j < NSUB; ++j) {
            const int row = c.wave * (16 * NSUB) + j * 16 + c.l16;
            const float s = (float)__builtin_bit_cast(_Float16, (uint16_t)(sc[j] >> (16 * bi)));
            const _Float16 sp1 = (_Float16)__builtin_amdgcn_ldexpf(s, c.negf);
            const half2v sp = {sp1, sp1};
            if (FMT == QL_FMT_INT8) {
                const int ch = (bi * 2 + (c.lg >> 1)) ^ ((row >> 2) & 3);
                const uint2 v = *reinterpret_cast<const uint2 *>(
                    stage + G::XBYTES + row * 64 + ch * 16 + (c.lg & 1) * 8);
                B[j] = deq_int8_f16(v.x, v.y, sp);
            } else {
                const int ch = bi ^ ((row >> 3) & 1);
                const uint32_t v = *reinterpret_cast<const uint32_t *>(
                    stage + G::XBYTES + row * 32 + ch * 16 + c.lg * 4);
                B[j] = deq_q4_f16(v, sp);
            }
        }
#pragma unroll
        for (int i = 0; i < MSUB; ++i) {
            const int row = i * 16 + c.l16;
            const int slot = bi * 512 + row * 4 + (c.lg ^ xswz(c.l16));
            const u32x4 a = *reinterpret_cast<const u32x4 *>(stage + slot * 16);
#pragma unroll
            for (int j = 0; j < NSUB; ++j)
                acc[i][j] = mfma_f16(a, B[j], acc[i][j]);
        }
    }
}

template <int FMT>
__device__ inline void compute_stage(const Ctx<FMT> &c, const uint8_t *stage,
                                     f32x4 (&acc)[MSUB][NSUB])
{
    using G = Geo<FMT>;
    constexpr bool OFFSET = FMT == QL_FMT_Q4;
    const u32x4 bneg = {0xC308C308u, 0xC308C308u, 0xC308C308u, 0xC308C308u};  // bf16 -136

    uint32_t sc[NSUB];
#pragma unroll
    for (int j = 0; j < NSUB; ++j)
        sc[j] = *reinterpret_cast<const uint32_t *>(stage + G::XBYTES + G::CBYTES +
                                                    (c.wave * (16 * NSUB) + j * 16 + c.l16) * 4);
#pragma unroll
    for (int bi = 0; bi < 2; ++bi) {
        u32x4 B[NSUB];
        float sf[NSUB];
#pragma unroll
        for (int j = 0; j < NSUB; ++j) {
            const int row = c.wave * (16 * NSUB) + j * 16 + c.l16;
            if (FMT == QL_FMT_INT8) {
                const int ch = (bi * 2 + (c.lg >> 1)) ^ ((row >> 2) & 3);
                const uint2 v = *reinterpret_cast<const uint2 *>(
                    stage + G::XBYTES + row * 64 + ch * 16 + (c.lg & 1) * 8);
                B[j] = cvt_int8(v.x, v.y);
            } else {
                const int ch = bi ^ ((row >> 3) & 1);
                const uint32_t v = *reinterpret_cast<const uint32_t *>(
                    stage + G::XBYTES + row * 32 + ch * 16 + c.lg * 4);
                B[j] = cvt_q4_off(v);
            }
            sf[j] = (float)__builtin_bit_cast(_Float16, (uint16_t)(sc[j] >> (16 * bi)));
        }
        // software pipeline over the row subtiles: the activation fragment of
        // subtile i+1 is read while subtile i's MFMAs run, and subtile i-1's
        // partials are scaled into the accumulators behind them; the
        // scheduling fences keep the compiler from hoisting every LDS read of
        // the step (which would exhaust the register file)
        auto read_a = [&](int i) {
            const int row = i * 16 + c.l16;
            const int slot = bi * 512 + row * 4 + (c.lg ^ xswz(row));
            return *reinterpret_cast<const u32x4 *>(stage + slot * 16);
        };
        u32x4 a = read_a(0);
        f32x4 P[NSUB], Pp[NSUB];
#pragma unroll
        for (int i = 0; i < MSUB; ++i) {
            const u32x4 an = i + 1 < MSUB ? read_a(i + 1) : a;
            f32x4 T = {0.f, 0.f, 0.f, 0.f};
            if (OFFSET)
                T = mfma(a, bneg, T);
#pragma unroll
            for (int j = 0; j < NSUB; ++j)
                P[j] = mfma(a, B[j], T);
            if (i > 0) {
#pragma unroll
                for (int j = 0; j < NSUB; ++j)
                    acc[i - 1][j] += sf[j] * Pp[j];
            }
#pragma unroll
            for (int j = 0; j < NSUB; ++j)
                Pp[j] = P[j];
            a = an;
            __builtin_amdgcn_sched_barrier(0);
        }
#pragma unroll
        for (int j = 0; j < NSUB; ++j)
            acc[MSUB - 1][j] += sf[j] * Pp[j];
    }
}

template <int FMT, bool F16>
__global__ __launch_bounds__(256, 2) void qgemm_big_kernel(const GroupArgs args)
{
    using G = Geo<FMT>;
    // one array per ring stage (distinct LDS objects)
    __shared__ __align__(16) uint8_t lds0[G::STAGE];
    __shared__ __align__(16) uint8_t lds1[G::STAGE];
    __shared__ __align__(16) uint8_t lds2[G::STAGE];
    uint8_t *const lds[NST] = {lds0, lds1, lds2};

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
    const int local = logical_tile(p - d.tile_begin, end - d.tile_begin);
    const int per_group = GROUP_M * d.tiles_n;
    const int gid = local / per_group;
    const int first_m = gid * GROUP_M;
    const int gsz = min(d.tiles_m - first_m, GROUP_M);
    const int within = local - gid * per_group;
    const int tm = first_m + within % gsz;
    const int tn = within / gsz;

    const int M = d.M, N = d.N, K = d.K, nb = K >> 5;
    const int m0 = tm * BM, n0 = tn * BN;
    const int tid = threadIdx.x;
    const int crow_bytes = FMT == QL_FMT_INT8 ? K : K / 2;

    Ctx<FMT> c;
    c.wave = tid >> 6;
    c.l16 = tid & 15;
    c.lg = (tid & 63) >> 4;
    c.xbase = reinterpret_cast<const uint8_t *>(d.X) + (int64_t)m0 * K * 2;
    c.cbase = d.codes + (int64_t)n0 * crow_bytes;
    c.sbase = reinterpret_cast<const uint8_t *>(d.scales) + (int64_t)n0 * nb * 2;
    // activations: stage slot = bi*512 + row*4 + (g ^ swz(row)); rows past M
    // repeat the last row (their outputs are never stored)
#pragma unroll
    for (int r = 0; r < G::XLOADS; ++r) {
        const int slot = r * 256 + tid;
        const int bi = slot >> 9, rem = slot & 511, row = rem >> 2;
        const int g = (rem & 3) ^ xswz(row);
        const int m = min(m0 + row, M - 1) - m0;
        c.xoff[r] = (uint32_t)(m * K * 2 + bi * 64 + g * 16);
    }
    // codes: stage slot = row*(CROW/16) + (chunk ^ swz(row)); rows past N
    // repeat the last row
#pragma unroll
    for (int r = 0; r < G::CLOADS; ++r) {
        const int slot = r * 256 + tid;
        int row, ch;
        if (FMT == QL_FMT_INT8) {
            row = slot >> 2;
            ch = (slot & 3) ^ ((row >> 2) & 3);
        } else {
            row = slot >> 1;
            ch = (slot & 1) ^ ((row >> 3) & 1);
        }
        const int n = min(n0 + row, N - 1) - n0;
        c.coff[r] = (uint32_t)(n * crow_bytes + ch * 16);
    }
    {
        // scales: one dword (blocks 2s, 2s+1) per weight row; surplus
        // wavefronts repeat the first rows (identical data, same slots), so
        // every wavefront issues the same number of loads per stage
        const int n = min(n0 + tid % BN, N - 1) - n0;
        c.soff = (uint32_t)(n * nb * 2);
    }

    f32x4 acc[MSUB][NSUB];
#pragma unroll
    for (int i = 0; i < MSUB; ++i)
#pragma unroll
        for (int j = 0; j < NSUB; ++j)
            acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    const int ns = nb >> 1;  // the host routes odd block counts elsewhere
    issue_stage<FMT>(c, lds[0], 0);
    if (ns > 1)
        issue_stage<FMT>(c, lds[1], 1);

    c.negf = 0;
    if (F16) {
        // largest scale of this tile's weight rows (fp16 bit patterns of
        // non-negative values compare as integers) -> shift keeping every
        // dequantized weight below 2^15 in magnitude.  Issued behind the
        // first two stages so its latency overlaps theirs.
        __shared__ uint32_t wmax[4];
        const int count = min(BN, N - n0) * nb / 2;  // dwords, contiguous
        const uint32_t *sp = reinterpret_cast<const uint32_t *>(c.sbase);
        uint32_t mx = 0;
        for (int q = tid; q < count; q += 256) {
            const uint32_t v = sp[q];
            mx = max(mx, max(v & 0x7FFFu, (v >> 16) & 0x7FFFu));
        }
#pragma unroll
        for (int o = 32; o >= 1; o >>= 1)
            mx = max(mx, (uint32_t)__shfl_xor((int)mx, o));
        if ((tid & 63) == 0)
            wmax[tid >> 6] = mx;
        // LDS write visible, then barrier (no fence: the ring stays in flight)
        __builtin_amdgcn_s_waitcnt(lgkm0_imm());
        __builtin_amdgcn_s_barrier();
        mx = max(max(wmax[0], wmax[1]), max(wmax[2], wmax[3]));
        const float smax = (float)__builtin_bit_cast(_Float16, (uint16_t)mx);
        if (smax > 0.f) {
            int E;
            (void)__builtin_frexpf(smax * (float)(FMT == QL_FMT_INT8 ? 127 : 7), &E);
            c.negf = 15 - E;  // Q * smax * 2^negf in [2^14, 2^15)
        }
    }

    // one step: wait for stage s (loads complete in issue order, so allowing
    // the LOADS youngest ones, which are stage s+1's, to remain outstanding
    // means all of stage s has landed), barrier, refill the slot that step
    // s-1 read with step s+2, compute stage s
#define QL_STEP(Q)                                                                  \
    {                                                                               \
        const int s = s0 + (Q);                                                     \
        if (s >= ns)                                                                \
            break;                                                                  \
        if (s + 1 < ns)                                                             \
            __builtin_amdgcn_s_waitcnt(vmcnt_imm(G::LOADS));                        \
        else                                                                        \
            __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));                               \
        __builtin_amdgcn_s_barrier();                                               \
        if (s + 2 < ns)                                                             \
            issue_stage<FMT>(c, lds[((Q) + 2) % NST], s + 2);                       \
        if (F16)                                                                    \
            compute_stage_f16<FMT>(c, lds[(Q)], acc);                               \
        else                                                                        \
            compute_stage<FMT>(c, lds[(Q)], acc);                                   \
    }

    for (int s0 = 0; s0 < ns; s0 += NST) {
        QL_STEP(0)
        QL_STEP(1)
        QL_STEP(2)
    }
#undef QL_STEP

    const int n_wave = n0 + c.wave * (16 * NSUB);
#pragma unroll
    for (int i = 0; i < MSUB; ++i)
#pragma unroll
        for (int j = 0; j < NSUB; ++j) {
            const int n = n_wave + j * 16 + c.l16;
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int m = m0 + i * 16 + c.lg * 4 + r;
                if (m < M && n < N)
                    d.Y[(int64_t)m * N + n] =
                        F16 ? __builtin_amdgcn_ldexpf(acc[i][j][r], d.xexp[m] - c.negf)
                            : acc[i][j][r];
            }
        }
}

}  // namespace

int big_tile_bm() { return BM; }
int big_tile_bn() { return BN; }

hipError_t launch_qgemm_big(int fmt, bool f16, const GroupArgs &args, hipStream_t stream)
{
    dim3 grid((unsigned)args.total_tiles), block(256);
    if (fmt == QL_FMT_INT8) {
        if (f16)
            hipLaunchKernelGGL((qgemm_big_kernel<QL_FMT_INT8, true>), grid, block, 0, stream, args);
        else
            hipLaunchKernelGGL((qgemm_big_kernel<QL_FMT_INT8, false>), grid, block, 0, stream, args);
    } else {
        if (f16)
            hipLaunchKernelGGL((qgemm_big_kernel<QL_FMT_Q4, true>), grid, block, 0, stream, args);
        else
            hipLaunchKernelGGL((qgemm_big_kernel<QL_FMT_Q4, false>), grid, block, 0, stream, args);
    }
    return hipGetLastError();
}

}  // namespace qlk
