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
// Decomposition.  A workgroup owns RW weight rows (8, 16, 32 or 64: NB =
// RW / 16 MFMA column blocks per wavefront, each activation fragment feeding
// all of them; with RW = 8 the MFMA's other 8 columns repeat the rows) and
// all M rows, for one of S parts of the K blocks.  The activation bytes a
// workgroup streams do not depend on RW, so wider row groups cut the
// activation re-reads (for 32 rows at K = 8192 they are 8x the codes of an
// 8-row group); the K parts restore the workgroup count.  Its KW wavefronts
// split the part's blocks in 8-block-aligned ranges, and their fp32 partial
// outputs are summed through LDS in wavefront order (deterministic).  With
// S > 1 each part stores a plain partial output part[S][M][N] that
// launch_split_sum adds up in part order.
//
// Contraction (exact, as in the other few-row path): per 32-wide block one
// v_mfma_f32_16x16x32_bf16 of the activation fragment against the codes in
// offset form (int8: byte ^ 0x80 = c + 128; q4: 0x4300 | (nibble ^ 8) =
// bf16(136 + c)), whose offset term -OFF * sum_{k in b} X[m][k] comes from a
// second MFMA against a constant -OFF matrix fed in as the C operand; the
// block's fp16 scale is then applied to the fp32 partial.
//
// Grouping.  One launch takes up to QL_MAX_GROUP layers of one format and
// row count (a DiT block's four linears): layer i owns the workgroups
// begin[i] .. begin[i + 1] - 1 of the grid, each layer with its own K parts;
// the template shape (rows per workgroup, wavefronts, activation stage) is
// common to the group.  All of a block's weights then stream in one launch,
// and its split layers share one sum launch.
//
// Requirements (checked by the host): K % 256 == 0, 16-byte aligned codes,
// scales and X.
#include <algorithm>
#include <cmath>

#include "epilogue.h"
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
    static constexpr int NB = RW >= 16 ? RW / 16 : 1;          // MFMA column blocks
    static constexpr int RL = RW >= 16 ? 16 : RW;               // rows per column block
    static constexpr int NSL = (RW + 15) / 16;                  // scale loads per 32 blocks
    static constexpr int BPC = 4;                               // blocks per chunk (128 k)
    static constexpr int CB = FMT == QL_FMT_INT8 ? 128 : 64;    // code bytes per row per chunk
    static constexpr int PPR = CB / 16;                         // 16-byte pieces per code row
    static constexpr int CODE = RW * CB;                        // code bytes per chunk
    static constexpr int XROW = 256;                            // activation bytes per row per chunk
    static constexpr int STAGE = CODE + MX * XROW;
    static constexpr int NCI = (CODE + 1023) / 1024;            // code loads per chunk
    static constexpr int NXI = MX * XROW / 1024;                // activation loads per chunk
    static constexpr int N = NCI + NXI;                         // loads per chunk (+NSL every 8)
    static constexpr int R = MX <= 8 ? 4 : 3;                   // ring depth (chunks)
    static constexpr int NF = MX / 16 > 1 ? MX / 16 : 1;        // 16-row activation fragments
    static constexpr int SLOT = RW * 64;                        // scales of 32 blocks
    static constexpr int WAVE = R * STAGE + 2 * SLOT;           // LDS bytes per wavefront
    static_assert((MX * XROW) % 1024 == 0, "whole activation loads");
    static_assert((R - 1) * N + NSL <= 63, "vmcnt range");
};

// code row j's physical 16-byte piece for logical piece p (bank spread for
// the fragment reads: int8 lanes read 8 bytes, q4 lanes 4 bytes)
template <int FMT>
__device__ inline int cswz(int j, int p)
{
    return FMT == QL_FMT_INT8 ? (p ^ ((j >> 1) & 7)) : (p ^ ((j >> 2) & 3));
}

// The kernel body for workgroup wg of layer d (the single-layer and the
// grouped kernel below differ only in how they find d: a single layer's
// descriptor is the whole kernel argument, so its fields load at once; a
// group's layer is looked up first)
template <int FMT, int RW, int MX, int KW>
__device__ __forceinline__ void stream_body(const LinDesc &d, const int wg)
{
    using G = SGeo<FMT, RW, MX>;
    __shared__ __align__(16) uint8_t lds[KW * G::WAVE];

    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int l16 = lane & 15, lg = lane >> 4;
    const int M = d.M, N = d.N, K = d.K, nb = K >> 5;
    // consecutive workgroups take the parts of one row group: with the
    // round-robin XCD dispatch, part p's activation range stays on few XCDs
    const int S = d.ksplit, part = wg % S;
    const int n0 = wg / S * RW;
    const int crow_bytes = FMT == QL_FMT_INT8 ? K : K / 2;

    uint8_t *const ring = lds + wave * G::WAVE;
    uint8_t *const sring = ring + G::R * G::STAGE;

    // this part's blocks [pb0, pb1) (psteps blocks, a multiple of 8), and
    // this wavefront's share [bw0, bw1), 8-aligned (whole scale pieces and
    // chunks; nb % 8 == 0)
    const int pb0 = min(part * d.psteps, nb), pb1 = min(pb0 + d.psteps, nb);
    const int per = (((pb1 - pb0 + KW - 1) / KW) + 7) & ~7;
    const int bw0 = min(pb0 + wave * per, pb1), bw1 = min(bw0 + per, pb1);
    const int nch = (bw1 - bw0) / G::BPC;

    // per-lane load offsets from wave-uniform 64-bit bases that advance per
    // chunk.  The bases hold the row group's first row n0, so a lane's
    // offset only spans the group's RW rows (< 64 K bytes; the host takes
    // this path for K <= 2^24 only, which keeps every offset below 2^31).
    uint32_t coff[G::NCI], xoff[G::NXI];
    bool cact[G::NCI];
#pragma unroll
    for (int r = 0; r < G::NCI; ++r) {
        const int o = (r * 64 + lane) * 16;  // byte offset in the chunk's code area
        const int j = o / G::CB, pp = (o % G::CB) / 16;
        cact[r] = j < RW;
        const int dn = min(n0 + min(j, RW - 1), N - 1) - n0;
        coff[r] = (uint32_t)(dn * crow_bytes + cswz<FMT>(j, pp) * 16);
    }
#pragma unroll
    for (int r = 0; r < G::NXI; ++r) {
        const int o = (r * 64 + lane) * 16;
        const int m = o / G::XROW, pp = (o % G::XROW) / 16;  // 16 pieces per row
        xoff[r] = (uint32_t)(min(m, M - 1) * K * 2 + (pp ^ (m & 15)) * 16);
    }
    // scales: lane -> (row j = 16 h + lane / 4, piece p = lane % 4) of a
    // 32-block run, h < NSL
    const int sp = lane & 3;

    const uint8_t *const cbase =
        d.codes + (int64_t)n0 * crow_bytes + (FMT == QL_FMT_INT8 ? bw0 * 32 : bw0 * 16);
    const uint8_t *const sbase8 =
        reinterpret_cast<const uint8_t *>(d.scales) + (int64_t)n0 * nb * 2;
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
        if (c % 8 == 0) {
            // scales of blocks bw0 + 4c .. + 31 (pieces past the row end
            // repeat its last piece; their values are never read)
            const int g = c / 8;
#pragma unroll
            for (int h = 0; h < G::NSL; ++h) {
                const int sj = 16 * h + (lane >> 2);
                const int dn = min(n0 + min(sj, RW - 1), N - 1) - n0;
                const int b = min(bw0 + 32 * g + 8 * ((sp ^ ((sj >> 2) & 3))), nb - 8);
                if (sj < RW)
                    dma16(sbase8, (uint32_t)(dn * nb * 2 + b * 2),
                          lds_addr(sring + (g & 1) * G::SLOT) + h * 1024);
            }
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
    f32x4 acc[G::NF][G::NB];
#pragma unroll
    for (int f = 0; f < G::NF; ++f)
#pragma unroll
        for (int nbi = 0; nbi < G::NB; ++nbi)
            acc[f][nbi] = f32x4{0.f, 0.f, 0.f, 0.f};
    const int jl = l16 % G::RL;  // weight row of this lane's MFMA column, block 0
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
            u32x4 B[G::NB];
            float sc[G::NB];
            // scale of block 4c + t (within the 32-block run of this chunk)
            const int bs = (c % 8) * 4 + t;  // 0..31
#pragma unroll
            for (int nbi = 0; nbi < G::NB; ++nbi) {
                const int j = nbi * 16 + jl;
                if (FMT == QL_FMT_INT8) {
                    // bytes [32 t + 8 lg, +8) of row j: logical piece 2t + lg/2
                    const int pp = cswz<FMT>(j, 2 * t + (lg >> 1));
                    const uint2 v = *reinterpret_cast<const uint2 *>(st + j * G::CB + pp * 16 +
                                                                     (lg & 1) * 8);
                    B[nbi] = cvt_int8_off(v.x, v.y);
                } else {
                    // bytes [16 t + 4 lg, +4) of row j: logical piece t
                    const int pp = cswz<FMT>(j, t);
                    const uint32_t v = *reinterpret_cast<const uint32_t *>(
                        st + j * G::CB + pp * 16 + lg * 4);
                    B[nbi] = cvt_q4_off(v);
                }
                const int spiece = (bs >> 3) ^ ((j >> 2) & 3);
                const uint16_t sbits = *reinterpret_cast<const uint16_t *>(
                    ss + j * 64 + spiece * 16 + (bs & 7) * 2);
                sc[nbi] = (float)__builtin_bit_cast(_Float16, sbits);
            }
#pragma unroll
            for (int f = 0; f < G::NF; ++f) {
                // activation fragment f: row f * 16 + mx, bf16 [32 t + 8 lg, +8) =
                // piece 4t + lg; its offset term is shared by the column blocks
                const int row = f * 16 + mx;
                const u32x4 a = *reinterpret_cast<const u32x4 *>(
                    st + G::CODE + row * G::XROW + ((4 * t + lg) ^ (row & 15)) * 16);
                const f32x4 off = mfma(a, bneg, f32x4{0.f, 0.f, 0.f, 0.f});
#pragma unroll
                for (int nbi = 0; nbi < G::NB; ++nbi)
                    acc[f][nbi] += sc[nbi] * mfma(a, B[nbi], off);
            }
        }
    }

    // sum the wavefronts' partial outputs in wavefront order (the ring
    // memory is reused once every wavefront is done with it)
    static_assert(G::NF * G::NB * KW * 64 * 16 <= KW * G::WAVE, "reduction fits the ring");
    __syncthreads();
    f32x4 *red = reinterpret_cast<f32x4 *>(lds);
#pragma unroll
    for (int f = 0; f < G::NF; ++f)
#pragma unroll
        for (int nbi = 0; nbi < G::NB; ++nbi)
            red[((f * G::NB + nbi) * KW + wave) * 64 + lane] = acc[f][nbi];
    __syncthreads();
    // destination: this part's partial output (summed, with the epilogue,
    // by a separate launch), or Y
    float *const Yd = S > 1 ? d.part + (int64_t)part * M * N : d.Y;
    // wavefront w sums (and stores) fragments (f, nbi) = w, w + KW, ...
    for (int q = wave; q < G::NF * G::NB; q += KW) {
        const int f = q / G::NB, nbi = q % G::NB;
        f32x4 y = red[(q * KW) * 64 + lane];
        for (int w = 1; w < KW; ++w)
            y += red[(q * KW + w) * 64 + lane];
        const int n = n0 + nbi * 16 + l16;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int m = f * 16 + lg * 4 + r;
            if (l16 < G::RL && m < M && n < N) {
                if (S > 1)
                    Yd[(int64_t)m * N + n] = y[r];
                else
                    epi_store(d.ep, d.Y, (int64_t)m * N + n, n, y[r]);
            }
        }
    }
}

template <int FMT, int RW, int MX, int KW>
__global__ __launch_bounds__(64 * KW) void qgemm_stream_kernel(const LinDesc d)
{
    stream_body<FMT, RW, MX, KW>(d, (int)blockIdx.x);
}

template <int FMT, int RW, int MX, int KW>
__global__ __launch_bounds__(64 * KW) void qgemm_stream_group_kernel(const LayerGroup grp)
{
    // this workgroup's layer (wave-uniform) and its index within the layer
    int li = 0;
    while (li + 1 < grp.n && (int)blockIdx.x >= grp.begin[li + 1])
        ++li;
    stream_body<FMT, RW, MX, KW>(grp.d[li], (int)blockIdx.x - grp.begin[li]);
}

template <int FMT, int RW, int MX, int KW>
hipError_t launch_kw(const LayerGroup &g, hipStream_t s)
{
    if constexpr (KW * SGeo<FMT, RW, MX>::WAVE > 160 * 1024) {
        return hipErrorInvalidValue;  // does not fit the LDS; never chosen
    } else {
        const dim3 grid((unsigned)g.begin[g.n]);
        if (g.n == 1)
            hipLaunchKernelGGL((qgemm_stream_kernel<FMT, RW, MX, KW>), grid, dim3(64 * KW), 0, s,
                               g.d[0]);
        else
            hipLaunchKernelGGL((qgemm_stream_group_kernel<FMT, RW, MX, KW>), grid, dim3(64 * KW),
                               0, s, g);
        return hipGetLastError();
    }
}

template <int FMT, int RW, int MX>
hipError_t launch_rw(int kw, const LayerGroup &g, hipStream_t s)
{
    switch (kw) {
    case 2: return launch_kw<FMT, RW, MX, 2>(g, s);
    case 4: return launch_kw<FMT, RW, MX, 4>(g, s);
    case 8: return launch_kw<FMT, RW, MX, 8>(g, s);
    default: return hipErrorInvalidValue;
    }
}

template <int FMT, int MX>
hipError_t launch_mx(int rw, int kw, const LayerGroup &g, hipStream_t s)
{
    switch (rw) {
    case 8: return launch_rw<FMT, 8, MX>(kw, g, s);
    case 16: return launch_rw<FMT, 16, MX>(kw, g, s);
    case 32: return launch_rw<FMT, 32, MX>(kw, g, s);
    case 64: return launch_rw<FMT, 64, MX>(kw, g, s);
    default: return hipErrorInvalidValue;
    }
}

template <int FMT>
hipError_t launch_fmt(const StreamPlan &p, const LayerGroup &g, hipStream_t s)
{
    switch (p.mx) {
    case 8: return launch_mx<FMT, 8>(p.rw, p.kw, g, s);
    case 16: return launch_mx<FMT, 16>(p.rw, p.kw, g, s);
    case 32: return launch_mx<FMT, 32>(p.rw, p.kw, g, s);
    default: return hipErrorInvalidValue;
    }
}

template <int FMT, int RW, int MX>
constexpr int wave_lds() { return SGeo<FMT, RW, MX>::WAVE; }

template <int FMT, int MX>
int geo(int rw, int &stage, int &ring)
{
    switch (rw) {
    case 8: stage = SGeo<FMT, 8, MX>::STAGE; ring = SGeo<FMT, 8, MX>::R; return wave_lds<FMT, 8, MX>();
    case 16: stage = SGeo<FMT, 16, MX>::STAGE; ring = SGeo<FMT, 16, MX>::R; return wave_lds<FMT, 16, MX>();
    case 32: stage = SGeo<FMT, 32, MX>::STAGE; ring = SGeo<FMT, 32, MX>::R; return wave_lds<FMT, 32, MX>();
    default: stage = SGeo<FMT, 64, MX>::STAGE; ring = SGeo<FMT, 64, MX>::R; return wave_lds<FMT, 64, MX>();
    }
}

// LDS bytes per wavefront, stage bytes and ring depth of a configuration
int stream_geo(int fmt, int mx, int rw, int &stage, int &ring)
{
    const bool i8 = fmt == QL_FMT_INT8;
    switch (mx) {
    case 8: return i8 ? geo<QL_FMT_INT8, 8>(rw, stage, ring) : geo<QL_FMT_Q4, 8>(rw, stage, ring);
    case 16: return i8 ? geo<QL_FMT_INT8, 16>(rw, stage, ring) : geo<QL_FMT_Q4, 16>(rw, stage, ring);
    default: return i8 ? geo<QL_FMT_INT8, 32>(rw, stage, ring) : geo<QL_FMT_Q4, 32>(rw, stage, ring);
    }
}

}  // namespace

int stream_max_m() { return 32; }
int stream_max_k() { return 1 << 24; }

// Choice of rows per workgroup, wavefronts and K parts for a group of
// layers (one format, one row count M).  Each wavefront keeps R - 1 chunks
// of loads in flight, so a workgroup streams its bytes (activations
// MX * Kp * 2, codes RW * Kp * cb for its part's Kp) in about
// bytes / (KW (R - 1) STAGE) memory round trips.  Every layer is cut into
// parts of about one common length (so that its workgroups take about as
// long as the others'); the launch takes as many workgroup rounds as the
// grid needs over the CUs, and a split adds the partial round trip and the
// sum launch.  No plan is faster than its total bytes (every workgroup
// reads the activations of its part, so few rows per workgroup re-read them
// more often) at the streaming rate.  The plan minimizes that estimate over
// the rows per workgroup, the wavefronts and the part length.
StreamPlan stream_plan(int fmt, const LinDesc *ds, int n, int cus, int *S, int *psteps)
{
    // fitted to a sweep of every plan on single layers and the grouped
    // d = 2048 block at M = 8, 16, 24 and 32, int8 and q4
    constexpr double RT = 2.5;           // us per memory round trip under load
    constexpr double SUM_LAUNCH = 3.0;   // us: split_sum launch and its gap
    constexpr double SUM_RATE = 4.0e6;   // bytes per us the sum launch moves
    constexpr double PART_COST = 0.3;    // us per part
    constexpr double STREAM_RATE = 7.0e6;  // bytes per us all workgroups stream together
    constexpr int MAXS = 16;
    int M = 0, nbmax = 0;
    for (int i = 0; i < n; ++i) {
        M = std::max(M, ds[i].M);
        nbmax = std::max(nbmax, ds[i].K / 32);
    }
    // at most 4 rows still stage 8: the 4-row stage's deeper ring measured
    // 15-25% slower on the d = 2048 block
    const int mx = M <= 8 ? 8 : M <= 16 ? 16 : 32;
    const double cb = fmt == QL_FMT_INT8 ? 1.0 : 0.5;
    StreamPlan best{mx, 16, 4, 1, nbmax};
    double best_t = 1e30;
    int bS[QL_MAX_GROUP], bP[QL_MAX_GROUP];
    for (int i = 0; i < n; ++i) {
        bS[i] = 1;
        bP[i] = ds[i].K / 32;
    }
    for (int rw : {8, 16, 32, 64}) {
        int stage = 0, ring = 0;
        const int wave = stream_geo(fmt, mx, rw, stage, ring);
        for (int kw : {2, 4, 8}) {
            if (kw * wave > 160 * 1024)
                continue;
            const int per_cu = std::min(160 * 1024 / (kw * wave), 2048 / (64 * kw));
            // part lengths (blocks): whole 8-block groups, >= 8 per
            // wavefront, doubling up to the longest layer's whole K
            int lens[16], nl = 0;
            for (int L = 8 * kw; L < nbmax && nl < 15; L *= 2)
                lens[nl++] = L;
            lens[nl++] = (nbmax + 7) & ~7;
            for (int li = 0; li < nl; ++li) {
                const int L = lens[li];
                int Si[QL_MAX_GROUP], Pi[QL_MAX_GROUP], Smax = 1;
                int64_t wgs = 0;
                double sum_bytes = 0.0, trips_max = 0.0, total_bytes = 0.0;
                bool ok = true;
                for (int i = 0; i < n && ok; ++i) {
                    const int nb = ds[i].K / 32;
                    int S = std::max(1, std::min(MAXS, (nb + L - 1) / L));
                    const int pb = ((nb + S - 1) / S + 7) & ~7;
                    S = (nb + pb - 1) / pb;
                    if (pb < 8 * kw)
                        ok = false;
                    Si[i] = S;
                    Pi[i] = pb;
                    Smax = std::max(Smax, S);
                    const int64_t wi = (int64_t)((ds[i].N + rw - 1) / rw) * S;
                    wgs += wi;
                    const double bytes = (double)pb * 32 * (mx * 2 + rw * cb);
                    total_bytes += (double)wi * bytes;
                    trips_max = std::max(trips_max,
                                         std::ceil(bytes / ((double)kw * (ring - 1) * stage)) + 1);
                    if (S > 1)
                        sum_bytes += (double)(S + 1) * ds[i].M * ds[i].N * 4;
                }
                if (!ok)
                    continue;
                const double rounds = std::ceil((double)wgs / ((double)cus * per_cu));
                double t = std::max(rounds * trips_max * RT, total_bytes / STREAM_RATE);
                if (Smax > 1)
                    t += RT + SUM_LAUNCH + sum_bytes / SUM_RATE + PART_COST * Smax;
                if (t < best_t * 0.97) {
                    best_t = t;
                    best = StreamPlan{mx, rw, kw, Smax, L};
                    std::copy(Si, Si + n, bS);
                    std::copy(Pi, Pi + n, bP);
                }
            }
        }
    }
    std::copy(bS, bS + n, S);
    std::copy(bP, bP + n, psteps);
    return best;
}

hipError_t launch_qgemm_stream(int fmt, const StreamPlan &p, const LayerGroup &g,
                               hipStream_t stream)
{
    return fmt == QL_FMT_INT8 ? launch_fmt<QL_FMT_INT8>(p, g, stream)
                              : launch_fmt<QL_FMT_Q4>(p, g, stream);
}

}  // namespace qlk
