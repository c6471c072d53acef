// Quantized linear forward for few activation rows (bf16, M <= 32):
// a weight-streaming kernel, bound by HBM bandwidth.
//
//   Y[m][n] = sum_b s[n][b] * sum_{k in b} X[m][k] * c[n][k]
//
// What limits such a kernel on this GPU is the number of memory requests
// rather than bytes: an MFMA-shaped load (16 weight rows x 8-32 bytes per
// instruction) costs one request per row for a fraction of a cache line.  So
// each wavefront streams its data with direct-to-LDS loads in whole lines --
// for its RW weight rows 128 bytes (int8) or 64 bytes (q4) of codes per row
// per chunk of 128 k, the matching 256-byte slices of the activation rows,
// and every 32 blocks one 64-byte run of each row's scales -- into an LDS
// ring of its own, and reads MFMA fragments from there.  The ring is private
// to the wavefront (it both issues the loads and consumes them), so no
// barrier is needed until the final reduction.
//
// Decomposition.  A workgroup owns RW weight rows (16; 8 when N is small, the
// MFMA's other 8 columns then repeat them) and all M rows; its KW wavefronts
// split the K blocks in 8-block-aligned ranges, and their fp32 partial
// outputs are summed through LDS in wavefront order (deterministic).
//
// Contraction (exact, as in the other few-row path): per 32-wide block one
// v_mfma_f32_16x16x32_bf16 of the activation fragment against the codes in
// offset form (int8: byte ^ 0x80 = c + 128; q4: 0x4300 | (nibble ^ 8) =
// bf16(136 + c)), whose offset term -OFF * sum_{k in b} X[m][k] comes from a
// second MFMA against a constant -OFF matrix fed in as the C operand; the
// block's fp16 scale is then applied to the fp32 partial.
//
// Requirements (checked by the host): K % 256 == 0, 16-byte aligned codes,
// scales and X.
#include "internal.h"

namespace qlk {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__device__ inline constexpr int vmcnt_imm(int v)
{
    // gfx9 s_waitcnt encoding: vmcnt[3:0] + vmcnt[5:4] at bits 15:14;
    // expcnt (bits 6:4) and lgkmcnt (bits 11:8) left at "no wait"
    return (v & 15) | (((v >> 4) & 3) << 14) | (7 << 4) | (15 << 8);
}

// wave-uniform 64-bit base in an SGPR pair (readfirstlane returns int:
// widen through uint32_t)
__device__ inline uint64_t sbase(const void *p)
{
    const uint64_t v = (uint64_t)(uintptr_t)p;
    const uint32_t lo = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)v);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)(v >> 32));
    return (uint64_t)lo | ((uint64_t)hi << 32);
}

// Direct-to-LDS 16-byte load: the active lane t's data lands at lds + t * 16.
__device__ inline void dma16(const void *base, uint32_t off, uint32_t lds)
{
    asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1"
                 :
                 : "v"(off), "s"(sbase(base)), "s"(__builtin_amdgcn_readfirstlane(lds))
                 : "memory");
}

__device__ inline uint32_t lds_addr(const void *p) { return (uint32_t)(uintptr_t)p; }

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
__device__ inline u32x4 cvt_int8_off(uint32_t lo, uint32_t hi)
{
    const uint32_t a = lo ^ 0x80808080u, b = hi ^ 0x80808080u;
    u32x4 r;
    r[0] = pack_hi((float)(a & 0xFF), (float)((a >> 8) & 0xFF));
    r[1] = pack_hi((float)((a >> 16) & 0xFF), (float)(a >> 24));
    r[2] = pack_hi((float)(b & 0xFF), (float)((b >> 8) & 0xFF));
    r[3] = pack_hi((float)((b >> 16) & 0xFF), (float)(b >> 24));
    return r;
}

// q4 codes (one dword, k0 in bits 0-3) -> bf16 of c + 136, natural order
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

template <int FMT, int RW, int MX>
struct SGeo {
    static constexpr int BPC = 4;                               // blocks per chunk (128 k)
    static constexpr int CB = FMT == QL_FMT_INT8 ? 128 : 64;    // code bytes per row per chunk
    static constexpr int PPR = CB / 16;                         // 16-byte pieces per code row
    static constexpr int CODE = RW * CB;                        // code bytes per chunk
    static constexpr int XROW = 256;                            // activation bytes per row per chunk
    static constexpr int STAGE = CODE + MX * XROW;
    static constexpr int NCI = (CODE + 1023) / 1024;            // code loads per chunk
    static constexpr int NXI = MX * XROW / 1024;                // activation loads per chunk
    static constexpr int N = NCI + NXI;                         // loads per chunk (+1 every 8)
    static constexpr int R = MX <= 4 ? 6 : MX <= 8 ? 4 : 3;     // ring depth (chunks)
    static constexpr int NF = MX / 16 > 1 ? MX / 16 : 1;        // 16-row activation fragments
    static constexpr int SLOT = RW * 64;                        // scales of 32 blocks
    static constexpr int WAVE = R * STAGE + 2 * SLOT;           // LDS bytes per wavefront
    static_assert((MX * XROW) % 1024 == 0, "whole activation loads");
    static_assert((R - 1) * N + 1 <= 63, "vmcnt range");
};

// code row j's physical 16-byte piece for logical piece p (bank spread for
// the fragment reads: int8 lanes read 8 bytes, q4 lanes 4 bytes)
template <int FMT>
__device__ inline int cswz(int j, int p)
{
    return FMT == QL_FMT_INT8 ? (p ^ ((j >> 1) & 7)) : (p ^ ((j >> 2) & 3));
}

template <int FMT, int RW, int MX, int KW>
__global__ __launch_bounds__(64 * KW) void qgemm_stream_kernel(const LinDesc d)
{
    using G = SGeo<FMT, RW, MX>;
    __shared__ __align__(16) uint8_t lds[KW * G::WAVE];

    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int l16 = lane & 15, lg = lane >> 4;
    const int M = d.M, N = d.N, K = d.K, nb = K >> 5;
    const int n0 = (int)blockIdx.x * RW;
    const int crow_bytes = FMT == QL_FMT_INT8 ? K : K / 2;

    uint8_t *const ring = lds + wave * G::WAVE;
    uint8_t *const sring = ring + G::R * G::STAGE;

    // this wavefront's blocks [bw0, bw1), 8-aligned (whole scale pieces and
    // chunks; nb % 8 == 0)
    const int per = (((nb + KW - 1) / KW) + 7) & ~7;
    const int bw0 = min(wave * per, nb), bw1 = min(bw0 + per, nb);
    const int nch = (bw1 - bw0) / G::BPC;

    // per-lane load offsets (from wave-uniform bases that advance per chunk)
    uint32_t coff[G::NCI], xoff[G::NXI], soff;
    bool cact[G::NCI];
#pragma unroll
    for (int r = 0; r < G::NCI; ++r) {
        const int o = (r * 64 + lane) * 16;  // byte offset in the chunk's code area
        const int j = o / G::CB, pp = (o % G::CB) / 16;
        cact[r] = j < RW;
        const int n = min(n0 + min(j, RW - 1), N - 1);
        coff[r] = (uint32_t)(n * crow_bytes + cswz<FMT>(j, pp) * 16);
    }
#pragma unroll
    for (int r = 0; r < G::NXI; ++r) {
        const int o = (r * 64 + lane) * 16;
        const int m = o / G::XROW, pp = (o % G::XROW) / 16;  // 16 pieces per row
        xoff[r] = (uint32_t)(min(m, M - 1) * K * 2 + (pp ^ (m & 15)) * 16);
    }
    // scales: lane -> (row j = lane / 4, piece p = lane % 4) of a 32-block run
    const int sj = lane >> 2, sp = lane & 3;
    const bool sact = sj < RW;
    const int srowi = min(n0 + min(sj, RW - 1), N - 1);

    const uint8_t *const cbase = d.codes + (FMT == QL_FMT_INT8 ? bw0 * 32 : bw0 * 16);
    const uint8_t *const xbase = reinterpret_cast<const uint8_t *>(d.X) + bw0 * 64;

    auto issue = [&](int c) {
        uint8_t *st = ring + (c % G::R) * G::STAGE;
#pragma unroll
        for (int r = 0; r < G::NCI; ++r)
            if (cact[r])
                dma16(cbase + c * G::CB, coff[r], lds_addr(st) + r * 1024);
#pragma unroll
        for (int r = 0; r < G::NXI; ++r)
            dma16(xbase + c * G::XROW, xoff[r], lds_addr(st + G::CODE) + r * 1024);
        if (c % 8 == 0 && sact) {
            // scales of blocks bw0 + 4c .. + 31 (pieces past the row end
            // repeat its last piece; their values are never read)
            const int g = c / 8;
            const int b = min(bw0 + 32 * g + 8 * ((sp ^ ((sj >> 2) & 3))), nb - 8);
            const uint8_t *sb = reinterpret_cast<const uint8_t *>(d.scales);
            dma16(sb, (uint32_t)(srowi * nb * 2 + b * 2), lds_addr(sring + (g & 1) * G::SLOT));
        }
    };

    // stage waits: all but the loads of the `younger` chunks issued after c
    auto wait_younger = [&](int younger) {
        switch (younger) {
        case 0: __builtin_amdgcn_s_waitcnt(vmcnt_imm(0)); break;
        case 1: __builtin_amdgcn_s_waitcnt(vmcnt_imm(1 * G::N)); break;
        case 2: __builtin_amdgcn_s_waitcnt(vmcnt_imm(2 * G::N)); break;
        case 3: __builtin_amdgcn_s_waitcnt(vmcnt_imm(3 * G::N)); break;
        case 4: __builtin_amdgcn_s_waitcnt(vmcnt_imm(4 * G::N)); break;
        default: __builtin_amdgcn_s_waitcnt(vmcnt_imm(5 * G::N)); break;
        }
    };

    const uint32_t negoff = FMT == QL_FMT_INT8 ? 0xC300C300u : 0xC308C308u;  // -128 / -136
    const u32x4 bneg = {negoff, negoff, negoff, negoff};
    f32x4 acc[G::NF];
#pragma unroll
    for (int f = 0; f < G::NF; ++f)
        acc[f] = f32x4{0.f, 0.f, 0.f, 0.f};
    const int j = l16 % RW;  // weight row of this lane's MFMA column
    // activation row of this lane's A fragment f: f * 16 + mx (rows >= M are
    // never stored; with MX < 16 the fragment's other rows repeat these)
    const int mx = l16 % (MX < 16 ? MX : 16);

#pragma unroll
    for (int c = 0; c < G::R - 1; ++c)
        if (c < nch)
            issue(c);
#pragma unroll 1
    for (int c = 0; c < nch; ++c) {
        if (c + G::R - 1 < nch)
            issue(c + G::R - 1);
        wait_younger(min(G::R - 1, nch - 1 - c));
        const uint8_t *st = ring + (c % G::R) * G::STAGE;
        const uint8_t *ss = sring + ((c / 8) & 1) * G::SLOT;
#pragma unroll
        for (int t = 0; t < G::BPC; ++t) {
            u32x4 B;
            if (FMT == QL_FMT_INT8) {
                // bytes [32 t + 8 lg, +8) of row j: logical piece 2t + lg/2
                const int pp = cswz<FMT>(j, 2 * t + (lg >> 1));
                const uint2 v = *reinterpret_cast<const uint2 *>(st + j * G::CB + pp * 16 +
                                                                 (lg & 1) * 8);
                B = cvt_int8_off(v.x, v.y);
            } else {
                // bytes [16 t + 4 lg, +4) of row j: logical piece t
                const int pp = cswz<FMT>(j, t);
                const uint32_t v = *reinterpret_cast<const uint32_t *>(st + j * G::CB + pp * 16 +
                                                                       lg * 4);
                B = cvt_q4_off(v);
            }
            // scale of block 4c + t (within the 32-block run of this chunk)
            const int bs = (c % 8) * 4 + t;  // 0..31
            const int spiece = (bs >> 3) ^ ((j >> 2) & 3);
            const uint16_t sbits = *reinterpret_cast<const uint16_t *>(
                ss + j * 64 + spiece * 16 + (bs & 7) * 2);
            const float s = (float)__builtin_bit_cast(_Float16, sbits);
#pragma unroll
            for (int f = 0; f < G::NF; ++f) {
                // activation fragment f: row f * 16 + mx, bf16 [32 t + 8 lg, +8) =
                // piece 4t + lg
                const int row = f * 16 + mx;
                const u32x4 a = *reinterpret_cast<const u32x4 *>(
                    st + G::CODE + row * G::XROW + ((4 * t + lg) ^ (row & 15)) * 16);
                acc[f] += s * mfma(a, B, mfma(a, bneg, f32x4{0.f, 0.f, 0.f, 0.f}));
            }
        }
    }

    // sum the wavefronts' partial outputs in wavefront order (the ring
    // memory is reused once every wavefront is done with it)
    __syncthreads();
    f32x4 *red = reinterpret_cast<f32x4 *>(lds);
#pragma unroll
    for (int f = 0; f < G::NF; ++f)
        red[(f * KW + wave) * 64 + lane] = acc[f];
    __syncthreads();
    if (wave == 0) {
#pragma unroll
        for (int f = 0; f < G::NF; ++f) {
            f32x4 y = red[f * KW * 64 + lane];
#pragma unroll
            for (int w = 1; w < KW; ++w)
                y += red[(f * KW + w) * 64 + lane];
            const int n = n0 + l16;
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int m = f * 16 + lg * 4 + r;
                if (l16 < RW && m < M && n < N)
                    d.Y[(int64_t)m * N + n] = y[r];
            }
        }
    }
}

template <int FMT, int RW, int MX, int KW>
hipError_t launch_kw(const LinDesc &d, hipStream_t s)
{
    if constexpr (KW * SGeo<FMT, RW, MX>::WAVE > 160 * 1024) {
        return hipErrorInvalidValue;  // does not fit the LDS; never chosen
    } else {
        const dim3 grid((unsigned)((d.N + RW - 1) / RW));
        hipLaunchKernelGGL((qgemm_stream_kernel<FMT, RW, MX, KW>), grid, dim3(64 * KW), 0, s, d);
        return hipGetLastError();
    }
}

template <int FMT, int RW, int MX>
hipError_t launch_rw(int kw, const LinDesc &d, hipStream_t s)
{
    switch (kw) {
    case 2: return launch_kw<FMT, RW, MX, 2>(d, s);
    case 4: return launch_kw<FMT, RW, MX, 4>(d, s);
    case 8: return launch_kw<FMT, RW, MX, 8>(d, s);
    default: return hipErrorInvalidValue;
    }
}

template <int FMT>
hipError_t launch_fmt(const LinDesc &d, hipStream_t s)
{
    // rows per workgroup: 16, or 8 when that would leave fewer workgroups
    // than CUs; wavefronts per workgroup: enough for ~2048 in the grid,
    // each with at least 16 blocks
    const int nb = d.K / 32;
    const bool narrow = (d.N + 15) / 16 < 256;
    const int groups = narrow ? (d.N + 7) / 8 : (d.N + 15) / 16;
    const int kw = (groups * 4 < 2048 && nb >= 8 * 16) ? 8 : 4;
    if (d.M <= 4)
        return narrow ? launch_rw<FMT, 8, 4>(kw, d, s) : launch_rw<FMT, 16, 4>(kw, d, s);
    if (d.M <= 8)
        return narrow ? launch_rw<FMT, 8, 8>(kw, d, s) : launch_rw<FMT, 16, 8>(kw, d, s);
    if (d.M <= 16)
        return narrow ? launch_rw<FMT, 8, 16>(kw, d, s) : launch_rw<FMT, 16, 16>(kw, d, s);
    // 32 activation rows: two wavefronts per workgroup keep two workgroups
    // per CU within the LDS; few row groups take four (one per CU)
    return narrow ? launch_rw<FMT, 8, 32>(4, d, s) : launch_rw<FMT, 16, 32>(2, d, s);
}

}  // namespace

int stream_max_m() { return 32; }

hipError_t launch_qgemm_stream(int fmt, const LinDesc &d, hipStream_t stream)
{
    return fmt == QL_FMT_INT8 ? launch_fmt<QL_FMT_INT8>(d, stream)
                              : launch_fmt<QL_FMT_Q4>(d, stream);
}

}  // namespace qlk
