// Quantized linear forward, large M, bf16 activations (the fp16 path):
//
//   Y[m][n] = sum_b s[n][b] * sum_{k in b} X[m][k] * c[n][k]
//
// computed as
//
//   Y[m][n] = 2^(e[m] - f[n]) * sum_k X'[m][k] * W'[n][k]
//   X'[m][k] = X[m][k] * 2^-e[m]                       (fp16, exact; xprep.hip)
//   W'[n][k] = fp16(c[n][k] * fp16(s[n][b] * 2^f[n]))   (one rounding)
//
// with the whole K accumulated in fp32 by v_mfma_f32_16x16x32_f16.  f[n] is
// chosen per weight row from the row's largest scale so that every |W'| is
// below 2^15: c is made exact in fp16 by a magic-number add (the fp16 bit
// pattern 0x6400 | u is 1024 + u) and one packed fp16 multiply by the scaled
// scale rounds c * s to 11 significant bits.  No per-block work remains on
// the accumulators, which is what made the exact per-block form
// (qgemm.hip: an fp32 FMA per output element per block) bound by VALU issue.
//
// Tile: 256 threads (4 wavefronts) compute BM x BN = 128 x 256 of Y.  Each
// wavefront owns a 128 x 64 strip (8 x 4 MFMA subtiles): every dequantized
// weight fragment feeds 8 MFMAs and every activation fragment 4.  The wide N
// extent halves the activation traffic per flop against a square tile: the
// fp16 activations (2 bytes per element, re-read once per column tile) are
// the larger operand stream next to 4-bit codes.
//
// Memory pipeline: activations, codes and scales move from global memory to
// LDS with the gfx950 direct-to-LDS loads (no VGPRs, no VALU), through a ring
// of NST stages of 64 k each (two scale blocks); a stage is issued NST - 1
// steps before it is consumed.  Each lane's offset within the tile is
// computed once; per step only the wave-uniform base (an SGPR pair)
// advances.  The loads are issued from inline asm so that the compiler's
// wait insertion, which cannot tell the ring stages apart and would drain
// every load in flight before each LDS read, stays out of the way: the
// kernel waits for each stage explicitly (s_waitcnt vmcnt, then s_barrier; a
// __syncthreads() would also drain the ring).  Nothing else here uses M0.
//
// LDS layouts are XOR-swizzled at 16-byte granularity so that fragment reads
// hit distinct banks.  A direct-to-LDS load writes lane t's data to slot
// base + t, so the swizzle is applied by choosing which global chunk each
// lane fetches.
//
// Tile order: within a layer, groups of 4 row tiles walked row-tile fastest;
// each of the 8 XCDs takes a contiguous range of one layer's tiles (L2
// reuse), and every layer of a grouped launch is spread over all XCDs.
#include "internal.h"

namespace qlk {
namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef _Float16 half2v __attribute__((ext_vector_type(2)));

constexpr int MSUB = 8, NSUB = 4, BM = 16 * MSUB, BN = 64 * NSUB, GROUP_M = 4;
constexpr int MAXSPLIT = 4;  // parts per output tile (split reduction)

template <int FMT>
struct Geo {
    static constexpr int NST = FMT == QL_FMT_INT8 ? 2 : 3;     // ring depth (LDS budget)
    static constexpr int XBYTES = BM * 64 * 2;                 // activations per stage
    static constexpr int CROW = FMT == QL_FMT_INT8 ? 64 : 32;  // code bytes per row per stage
    static constexpr int CBYTES = BN * CROW;
    static constexpr int STAGE = XBYTES + CBYTES;
    // scales travel apart: one 16-byte chunk (8 blocks = 4 steps) per weight
    // row every 4 steps, into a 2-slot ring; a per-step load would cost one
    // memory request per row for 4 bytes
    static constexpr int SGROUP = 4, SSLOT = BN * 16;
    static constexpr int XLOADS = XBYTES / 16 / 256;
    static constexpr int CLOADS = CBYTES / 16 / 256;
    static constexpr int LOADS = XLOADS + CLOADS;  // direct-to-LDS loads per step (+1 every 4)
    static constexpr int LDS = NST * STAGE + 2 * SSLOT;
    static_assert(XBYTES % (16 * 256) == 0 && CBYTES % (16 * 256) == 0,
                  "every thread issues the same number of 16-byte loads per stage");
    static_assert(BN == 256, "one scale chunk per weight row per thread");
    static_assert(2 * LDS <= 160 * 1024, "two workgroups per CU");
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

// Direct-to-LDS loads from (wave-uniform base + per-lane 32-bit offset):
// lane t's data lands at LDS address lds + t * size.
// The base is wave-uniform by construction; readfirstlane makes that
// visible to the compiler so it always lands in an SGPR pair.
__device__ inline uint64_t sbase(const void *p)
{
    const uint64_t v = (uint64_t)(uintptr_t)p;
    // readfirstlane returns int: widen through uint32_t (no sign extension)
    const uint32_t lo = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)v);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)(v >> 32));
    return (uint64_t)lo | ((uint64_t)hi << 32);
}

__device__ inline void dma16(const void *base, uint32_t off, uint32_t lds)
{
    asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1"
                 :
                 : "v"(off), "s"(sbase(base)), "s"(__builtin_amdgcn_readfirstlane(lds))
                 : "memory");
}

__device__ inline uint32_t lds_addr(const void *p)
{
    // a generic pointer into LDS carries the LDS offset in its low 32 bits
    return (uint32_t)(uintptr_t)p;
}

__device__ inline f32x4 mfma_f16(u32x4 a, u32x4 b, f32x4 c)
{
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(half8, a),
                                                  __builtin_bit_cast(half8, b), c, 0, 0, 0);
}

__device__ inline uint32_t h2mul_add(uint32_t v, half2v bias, half2v sp)
{
    // (v + bias) is exact (an fp16 integer), then one rounded multiply
    return __builtin_bit_cast(uint32_t, (__builtin_bit_cast(half2v, v) + bias) * sp);
}

// 8 int8 codes -> 8 fp16 of c * s', natural order.  byte ^ 0x80 = c + 128 is
// placed under the fp16 pattern 0x64 (= 1024 + (c + 128)) by v_perm; adding
// -1152 leaves c exactly.
__device__ inline u32x4 deq_int8(uint32_t a, uint32_t b, half2v sp)
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

// 8 q4 codes (k0 in bits 0-3) -> 8 fp16 of c * s', natural order: byte j of
// x holds codes 2j and 2j+1; v_perm puts byte j of x and of x >> 4 in the two
// 16-bit halves, the AND keeps one nibble (u = c + 8) in each and the OR
// sets the fp16 pattern 0x6400 | u = 1024 + u; adding -1032 leaves c.
__device__ inline u32x4 deq_q4(uint32_t c, half2v sp)
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

// 16-byte store / load at device coherence (write-through to, and read
// from, the level shared by all XCDs)
__device__ inline void st_coherent(float *p, f32x4 v)
{
    asm volatile("global_store_dwordx4 %0, %1, off sc1" : : "v"(p), "v"(v) : "memory");
}

__device__ inline f32x4 ld_coherent(const float *p)
{
    f32x4 v;
    asm volatile("global_load_dwordx4 %0, %1, off sc1" : "=v"(v) : "v"(p) : "memory");
    return v;
}

// wait for every load issued above; the values pass through the statement so
// that no use can be scheduled before it
template <int A, int B>
__device__ inline void wait_loads(f32x4 (&v)[A][B])
{
    static_assert(A * B == 12, "operand list below");
    asm volatile("s_waitcnt vmcnt(0)"
                 : "+v"(v[0][0]), "+v"(v[0][1]), "+v"(v[0][2]), "+v"(v[0][3]),
                   "+v"(v[1][0]), "+v"(v[1][1]), "+v"(v[1][2]), "+v"(v[1][3]),
                   "+v"(v[2][0]), "+v"(v[2][1]), "+v"(v[2][2]), "+v"(v[2][3])
                 :
                 : "memory");
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
    uint8_t *sring;  // the scale ring (2 slots of BN rows x 16 bytes)
    int wave, l16, lg;
    int f[NSUB];  // weight row (wave * 64 + j * 16 + l16) enters as W * 2^f[j]
};

// Issue the direct-to-LDS loads of step s into one ring stage (and, every
// SGROUP steps, the scales of steps s .. s + 3 into their ring slot).
template <int FMT>
__device__ inline void issue_stage(const Ctx<FMT> &c, uint8_t *stage, int s)
{
    using G = Geo<FMT>;
    const uint32_t base = lds_addr(stage);
    const uint8_t *xb = c.xbase + s * 128;  // 64 fp16 per row per step
    const uint8_t *cb = c.cbase + s * G::CROW;
#pragma unroll
    for (int r = 0; r < G::XLOADS; ++r)
        dma16(xb, c.xoff[r], base + (r * 256 + c.wave * 64) * 16);
#pragma unroll
    for (int r = 0; r < G::CLOADS; ++r)
        dma16(cb, c.coff[r], base + G::XBYTES + (r * 256 + c.wave * 64) * 16);
    if (s % G::SGROUP == 0) {
        const int g = s / G::SGROUP;
        dma16(c.sbase + g * 16, c.soff,
              lds_addr(c.sring + (g & 1) * G::SSLOT) + c.wave * 64 * 16);
    }
}

// fp16 pair {s * 2^f, s * 2^f} for the scale in the low half of v
__device__ inline half2v scaled_pair(uint32_t v, int f)
{
    const _Float16 s = __builtin_amdgcn_ldexph(__builtin_bit_cast(_Float16, (uint16_t)v), f);
    return half2v{s, s};
}

template <int FMT>
__device__ inline void compute_stage(const Ctx<FMT> &c, const uint8_t *stage, int s,
                                     f32x4 (&acc)[MSUB][NSUB])
{
    using G = Geo<FMT>;
    // scales of blocks 2s, 2s+1: dword s % 4 of the row's chunk in slot (s / 4) & 1
    const uint8_t *ss = c.sring + ((s / G::SGROUP) & 1) * G::SSLOT + (s % G::SGROUP) * 4;
    uint32_t sc[NSUB];
#pragma unroll
    for (int j = 0; j < NSUB; ++j)
        sc[j] = *reinterpret_cast<const uint32_t *>(ss + (c.wave * 64 + j * 16 + c.l16) * 16);
#pragma unroll
    for (int bi = 0; bi < 2; ++bi) {
        u32x4 B[NSUB];
#pragma unroll
        for (int j = 0; j < NSUB; ++j) {
            const int row = c.wave * 64 + j * 16 + c.l16;
            const half2v sp = scaled_pair(sc[j] >> (16 * bi), c.f[j]);
            if (FMT == QL_FMT_INT8) {
                const int ch = (bi * 2 + (c.lg >> 1)) ^ ((row >> 2) & 3);
                const uint2 v = *reinterpret_cast<const uint2 *>(
                    stage + G::XBYTES + row * 64 + ch * 16 + (c.lg & 1) * 8);
                B[j] = deq_int8(v.x, v.y, sp);
            } else {
                const int ch = bi ^ ((row >> 3) & 1);
                const uint32_t v = *reinterpret_cast<const uint32_t *>(
                    stage + G::XBYTES + row * 32 + ch * 16 + c.lg * 4);
                B[j] = deq_q4(v, sp);
            }
        }
#pragma unroll
        for (int i = 0; i < MSUB; ++i) {
            const int slot = bi * 512 + (i * 16 + c.l16) * 4 + (c.lg ^ xswz(c.l16));
            const u32x4 a = *reinterpret_cast<const u32x4 *>(stage + slot * 16);
#pragma unroll
            for (int j = 0; j < NSUB; ++j)
                acc[i][j] = mfma_f16(a, B[j], acc[i][j]);
        }
    }
}

template <int FMT>
__global__ __launch_bounds__(256, 2) void qgemm_wide_kernel(const GroupArgs args)
{
    using G = Geo<FMT>;
    constexpr int NST = G::NST, PD = NST - 1;  // prefetch distance in steps
    __shared__ __align__(16) uint8_t ring[G::LDS];

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
    // the ksplit parts of one output tile are adjacent (same XCD)
    const int local = logical_tile(p - d.tile_begin, end - d.tile_begin);
    const int S = d.ksplit;
    const int tile = local / S, part = local - tile * S;
    const int per_group = GROUP_M * d.tiles_n;
    const int gid = tile / per_group;
    const int first_m = gid * GROUP_M;
    const int gsz = min(d.tiles_m - first_m, GROUP_M);
    const int within = tile - gid * per_group;
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
    // scales: one 16-byte chunk of weight row tid per 4 steps
    c.soff = (uint32_t)((min(n0 + tid, N - 1) - n0) * nb * 2);
    c.sring = ring + NST * G::STAGE;

    // this part's steps of 64 k: [s0, s0 + ns); s0 is a multiple of the
    // scale group (psteps % 4 == 0, checked by the host)
    const int s0 = part * d.psteps;
    const int ns = min(nb >> 1, s0 + d.psteps) - s0;
    c.xbase += s0 * 128;
    c.cbase += s0 * G::CROW;
    c.sbase += s0 / G::SGROUP * 16;
#pragma unroll
    for (int q = 0; q < PD; ++q)
        if (q < ns)
            issue_stage<FMT>(c, ring + q * G::STAGE, q);

    // Row shifts, behind the first stages so their latency overlaps: lane
    // (l16, lg) scans a quarter of the scales of each of its NSUB weight rows
    // (16-byte chunks lg, lg + 4, ...; K % 256 == 0 and 16-byte aligned
    // scales, checked by the host); the four quarters are then combined.
    // fp16 bit patterns of non-negative values order as integers.
#pragma unroll
    for (int j = 0; j < NSUB; ++j) {
        const int n = min(n0 + c.wave * 64 + j * 16 + c.l16, N - 1);
        const u32x4 *srow = reinterpret_cast<const u32x4 *>(d.scales + (int64_t)n * nb);
        uint32_t mx = 0;
        for (int q = c.lg; q < nb / 8; q += 4) {
            const u32x4 v = srow[q];
#pragma unroll
            for (int t = 0; t < 4; ++t)
                mx = max(mx, max(v[t] & 0x7FFFu, (v[t] >> 16) & 0x7FFFu));
        }
        mx = max(mx, (uint32_t)__shfl_xor((int)mx, 16));
        mx = max(mx, (uint32_t)__shfl_xor((int)mx, 32));
        const float smax = (float)__builtin_bit_cast(_Float16, (uint16_t)mx);
        int E = 0;
        (void)__builtin_frexpf(smax * (float)(FMT == QL_FMT_INT8 ? 127 : 7), &E);
        c.f[j] = mx ? 15 - E : 0;  // Q * smax * 2^f in [2^14, 2^15)
    }

    f32x4 acc[MSUB][NSUB];
#pragma unroll
    for (int i = 0; i < MSUB; ++i)
#pragma unroll
        for (int j = 0; j < NSUB; ++j)
            acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    // one step: wait for stage s (loads complete in issue order, so allowing
    // the loads of the younger stages already issued to remain outstanding
    // means all of stage s has landed), barrier (every wavefront is done with
    // the slot step s-1 read), refill that slot with step s+PD, compute s
    static_assert(PD == 1 || PD == 2, "wait counts cover one or two stages in flight");
    int slot = 0;
#pragma unroll 1
    for (int s = 0; s < ns; ++s) {
        // stage s+1's loads (one more when it starts a scale group) may
        // remain in flight
        if (PD == 2 && s + 1 < ns && (s + 1) % G::SGROUP == 0)
            __builtin_amdgcn_s_waitcnt(vmcnt_imm(G::LOADS + 1));
        else if (PD == 2 && s + 1 < ns)
            __builtin_amdgcn_s_waitcnt(vmcnt_imm(G::LOADS));
        else
            __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));
        __builtin_amdgcn_s_barrier();
        const int fill = slot + PD >= NST ? slot + PD - NST : slot + PD;
        if (s + PD < ns)
            issue_stage<FMT>(c, ring + fill * G::STAGE, s + PD);
        compute_stage<FMT>(c, ring + slot * G::STAGE, s, acc);
        slot = slot + 1 == NST ? 0 : slot + 1;
    }

    // back to the scale of X * W^T (exact power-of-two factors)
#pragma unroll
    for (int i = 0; i < MSUB; ++i)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int m = min(m0 + i * 16 + c.lg * 4 + r, M - 1);
            const int e = d.xexp[m];
#pragma unroll
            for (int j = 0; j < NSUB; ++j)
                acc[i][j][r] = __builtin_amdgcn_ldexpf(acc[i][j][r], e - c.f[j]);
        }

    if (S > 1) {
        // Split reduction: publish this part's partial tile, count the
        // arrival; the last part to arrive adds all partials in part order
        // (the same sum whichever part finishes last).  A partial tile is
        // stored thread-major (each thread's 16-byte accumulator groups,
        // consecutive across the wavefront) with device-coherent
        // write-through stores and read back with device-coherent loads (the
        // parts of a tile may run on different XCDs, whose L2s are not
        // coherent); the stores are complete (s_waitcnt vmcnt(0)) before the
        // arrival is counted.  A release/acquire fence pair would instead
        // write back and invalidate each XCD's whole L2.
        float *const tp = d.part + (int64_t)tile * S * (BM * BN);
        float *const mine = tp + (int64_t)part * (BM * BN);
#pragma unroll
        for (int i = 0; i < MSUB; ++i)
#pragma unroll
            for (int j = 0; j < NSUB; ++j)
                st_coherent(mine + ((i * NSUB + j) * 256 + tid) * 4, acc[i][j]);
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        __syncthreads();  // the tile's stores are complete; the ring is no longer read
        int *const flag = reinterpret_cast<int *>(ring);
        if (tid == 0)
            *flag = __hip_atomic_fetch_add(d.cnt + tile, 1, __ATOMIC_RELAXED,
                                           __HIP_MEMORY_SCOPE_AGENT);
        __syncthreads();
        if (*flag != S - 1)
            return;
#pragma unroll
        for (int i = 0; i < MSUB; ++i) {
            // the other parts' groups of row block i, all in flight at once
            f32x4 v[MAXSPLIT - 1][NSUB];
#pragma unroll
            for (int q = 0; q < MAXSPLIT - 1; ++q) {
                const int qq = q < part ? q : q + 1;
#pragma unroll
                for (int j = 0; j < NSUB; ++j)
                    if (qq < S)
                        v[q][j] = ld_coherent(tp + (int64_t)qq * (BM * BN) +
                                              ((i * NSUB + j) * 256 + tid) * 4);
            }
            wait_loads(v);
#pragma unroll
            for (int j = 0; j < NSUB; ++j) {
                f32x4 y = part == 0 ? acc[i][j] : v[0][j];
#pragma unroll
                for (int q = 1; q < MAXSPLIT; ++q)
                    if (q < S)
                        y += q == part ? acc[i][j] : v[q < part ? q : q - 1][j];
                acc[i][j] = y;
            }
        }
        // fall through: the summed tile is stored like an unsplit one
    }

#pragma unroll
    for (int i = 0; i < MSUB; ++i)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int m = m0 + i * 16 + c.lg * 4 + r;
            if (m >= M)
                continue;
#pragma unroll
            for (int j = 0; j < NSUB; ++j) {
                const int n = n0 + c.wave * 64 + j * 16 + c.l16;
                if (n < N)
                    d.Y[(int64_t)m * N + n] = acc[i][j][r];
            }
        }
}

}  // namespace

int wide_tile_bm() { return BM; }
int wide_tile_bn() { return BN; }
int wide_max_split() { return MAXSPLIT; }

hipError_t launch_qgemm_wide(int fmt, const GroupArgs &args, hipStream_t stream)
{
    dim3 grid((unsigned)args.total_tiles), block(256);
    if (fmt == QL_FMT_INT8)
        hipLaunchKernelGGL(qgemm_wide_kernel<QL_FMT_INT8>, grid, block, 0, stream, args);
    else
        hipLaunchKernelGGL(qgemm_wide_kernel<QL_FMT_Q4>, grid, block, 0, stream, args);
    return hipGetLastError();
}

}  // namespace qlk
