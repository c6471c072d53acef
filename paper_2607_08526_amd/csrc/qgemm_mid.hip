// Quantized linear forward for a few hundred activation rows (bf16 X, int8
// or q4 weights; the dispatch sends 32 < M <= mid_max_m() here):
//
//   Y[m][n] = sum_b s[n][b] * sum_{k in b} X[m][k] * c[n][k]
//
// in its exact per-block form, in one launch with no activation pre-pass.
//
// Why a kernel of its own.  At a few hundred rows the work of a layer is a
// few GFLOP: spread over 256 CUs it is a handful of 64-k steps per workgroup,
// so what decides the time is the fixed cost around the product (launches,
// the first stage's memory latency, split partials), not the matrix-core
// rate.  The large-M kernel needs a pass over every activation row first (its
// fp16 activation copy and row shifts) and, with its 128 x 256 tiles, many K
// parts whose fp32 partials outweigh the 4-bit weights several times over.
// Here the bf16 activations are the MFMA operand as they are, the tile is
// 128 x 128 (twice the tiles, so half the K parts), and the block scale is
// applied in fp32 to each block's partial sum.
//
// Numerics (as in the other exact kernels).  Per 32-k block and 32 x 32
// output tile, two v_mfma_f32_32x32x16_bf16 form the block's partial sum
// from the bf16 activations and the codes in offset form, exact in bf16:
//   int8: byte ^ 0x80 = c + 128, converted by v_cvt_f32_ubyteN
//   q4:   nibble ^ 8 = c + 8 under the bf16 pattern 0x4300 (= 128): 136 + c
// The offset's contribution -OFF * sum_{k in b} X[m][k] is one more pair of
// MFMAs per row block and block (the activation fragments against a
// constant -OFF matrix), shared by the wavefront's column blocks and fed to
// their first MFMA as the C operand; the partial that leaves the second
// MFMA is offset-free, and acc += s[n][b] * partial applies the fp16 scale
// in fp32.
//
// k order.  Within a step of 64 k (two scale blocks), lane group g = l / 32
// of the 16-k chunk h of block b holds k = 32 b + 16 g + 8 h + e (e = 0..7):
// each MFMA stays inside one block, and a lane's codes of a block are one
// contiguous run (16 bytes int8, 8 bytes q4).
//
// MFMA layout (32 x 32 x 16): lane l holds A[l % 32][8 (l / 32) + e] and
// B[8 (l / 32) + e][l % 32]; accumulator register r of lane l is
// D[8 (r / 4) + 4 (l / 32) + r % 4][l % 32].
//
// Tile: 256 threads = 4 wavefronts in a 2 x 2 arrangement, each owning a 64
// x 64 quarter of the 128 x 128 output tile (2 x 2 MFMA tiles): every
// converted weight fragment feeds two MFMAs, every activation fragment two,
// and the offset pair is shared by the two column blocks.
//
// Memory pipeline (as in the large-M kernel): activations and codes move to
// LDS with direct-to-LDS loads (no VGPRs) through a ring of NST = 3 64-k
// stages; the weight rows' scales move one 16-byte chunk (8 blocks = 4
// steps) per row every 4 steps into a ring of SRING slots.  A 128-row tile has
// half as many scale chunks as threads: the upper half of the threads fetch
// the same chunks again into the unused half of the slot, so that every
// thread issues the same loads (the stage waits count loads per thread).
// Each stage is waited for explicitly (s_waitcnt vmcnt, then s_barrier) and
// the slot read in the previous step is refilled right after the barrier,
// NST - 1 steps ahead.  LDS layouts are XOR-swizzled at 16-byte granularity so
// that fragment reads are free of bank conflicts.
//
// Decomposition: a launch takes up to QL_MAX_GROUP layers (a DiT block's
// linears); each layer's tiles (row tiles fastest, so the row tiles of one
// weight strip share an XCD's L2) may be cut into K parts, adjacent in the
// launch; parts store plain fp32 partial outputs part[S][M][N] that
// launch_split_sum adds in part order (and applies the layer's epilogue
// to).  (Adding the parts in the kernel, by the last part to arrive at a
// tile, measured slower here: the device-coherent partial stores, the
// arrival and the last arriver's reloads serialize several memory round
// trips at the end of every split tile.)  A layer in one part applies its
// epilogue at the store.
//
// Requirements (checked by the host, mid_fits): K % 256 == 0, K < 2^23,
// 16-byte aligned X, codes and scales; psteps % 4 == 0.
#include <algorithm>
#include <type_traits>

#include "epilogue.h"
#include "internal.h"

namespace qlk {
namespace {

typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

constexpr int THREADS = 256, BM = 128, BN = 128;
constexpr int SGROUP = 4;  // steps per scale chunk
// Ring depth and resident workgroups per CU: three stages (two ahead of the
// one being read) and two workgroups per CU, whose wavefronts fill each
// other's stalls.  (Measured on the 128-row and 214-row workloads: deeper
// rings at one workgroup per CU, and eight wavefronts splitting each step's
// two blocks, were no faster.)
#ifndef QL_MID_NST
#define QL_MID_NST 3
#endif
#ifndef QL_MID_WGS
#define QL_MID_WGS 2
#endif
constexpr int NST = QL_MID_NST, WGS = QL_MID_WGS;
// Scale chunks: the chunk of steps 4 q .. 4 q + 3 is issued with stage 4 q,
// NST - 1 steps ahead, into slot q % SRING; the slot's previous chunk
// (steps 4 (q - SRING) .. + 3) must be finished by then.
constexpr int SRING = (NST + 2) / SGROUP + 1;
static_assert(SGROUP * (SRING - 1) - 3 > NST - 1 - SGROUP, "scale slot reuse");

template <int FMT>
struct MidGeo {
    static constexpr int XBYTES = BM * 128;                       // 64 bf16 per row
    static constexpr int CROW = FMT == QL_FMT_INT8 ? 64 : 32;     // code bytes per row
    static constexpr int CCH = CROW / 16;                         // 16-byte chunks per row
    static constexpr int CBYTES = BN * CROW;
    static constexpr int STAGE = XBYTES + CBYTES;
    static constexpr int SSLOT = THREADS * 16;                    // scale chunks (upper half unused)
    static constexpr int XLOADS = XBYTES / 16 / THREADS;
    static constexpr int CLOADS = CBYTES / 16 / THREADS;
    static constexpr int LOADS = XLOADS + CLOADS;                 // per thread and stage
    static constexpr int LDS = NST * STAGE + SRING * SSLOT;
    static constexpr uint32_t OFFW = FMT == QL_FMT_INT8 ? 0xC300C300u : 0xC308C308u;  // -OFF
    static_assert(XBYTES % (16 * THREADS) == 0 && CBYTES % (16 * THREADS) == 0,
                  "every thread issues the same number of 16-byte loads per stage");
    static_assert(WGS * LDS <= 160 * 1024, "resident workgroups per CU");
};

__device__ inline constexpr int vmcnt_imm(int v)
{
    // gfx9 s_waitcnt encoding: vmcnt[3:0] + vmcnt[5:4] at bits 15:14;
    // expcnt (bits 6:4) and lgkmcnt (bits 11:8) left at "no wait"
    return (v & 15) | (((v >> 4) & 3) << 14) | (7 << 4) | (15 << 8);
}

// physical 16-byte chunk = logical ^ swizzle(row)
__device__ inline int xswz(int row) { return (row & 7) ^ ((row >> 3) & 1); }
template <int FMT>
__device__ inline int cswz(int row)
{
    return FMT == QL_FMT_INT8 ? ((row >> 1) ^ (row >> 3)) & 3 : ((row >> 2) ^ (row >> 3)) & 1;
}

// wave-uniform 64-bit base in an SGPR pair (readfirstlane returns int: widen
// through uint32_t)
__device__ inline uint64_t sbase(const void *p)
{
    const uint64_t v = (uint64_t)(uintptr_t)p;
    const uint32_t lo = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)v);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)(v >> 32));
    return (uint64_t)lo | ((uint64_t)hi << 32);
}

// Direct-to-LDS 16-byte load from (wave-uniform base + per-lane offset):
// lane t's data lands at lds + t * 16.
__device__ inline void dma16(const void *base, uint32_t off, uint32_t lds)
{
    asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1"
                 :
                 : "v"(off), "s"(sbase(base)), "s"(__builtin_amdgcn_readfirstlane(lds))
                 : "memory");
}

__device__ inline uint32_t lds_addr(const void *p) { return (uint32_t)(uintptr_t)p; }

__device__ inline f32x16 mfma(u32x4 a, u32x4 b, f32x16 c)
{
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a),
                                                   __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

__device__ inline int logical_tile(int p, int G)
{
    // hardware places workgroup p on XCD p % 8; each XCD takes a contiguous
    // range of the logical order (XCDs 0..r-1 take q+1, the rest q)
    const int q = G >> 3, r = G & 7;
    const int xcd = p & 7, idx = p >> 3;
    return xcd < r ? xcd * (q + 1) + idx : r * (q + 1) + (xcd - r) * q + idx;
}

// An empty statement that the compiler keeps in order with the scheduling
// barriers: a value passed through it is computed in the MFMA group it is
// written in.  (Without it the optimizer moves MFMAs, fragment reads and
// scale FMAs next to their uses, and the block partials of a whole step end
// up live at once.)
template <typename T>
__device__ inline void pin(T &v)
{
    asm volatile("" : "+v"(v));
}

// 8 codes (k0..k7 of one 16-k chunk half) -> bf16 pairs (k0,k1) .. (k6,k7)
// of c + OFF.
//   int8: two dwords, byte i = code k_i
__device__ inline uint32_t bf16_pair(float lo, float hi)
{
    // integers < 256: the bf16 pattern is the fp32 pattern's high half
    return __builtin_amdgcn_perm(__float_as_uint(hi), __float_as_uint(lo), 0x07060302u);
}
__device__ inline u32x4 cvt_int8(uint32_t w0, uint32_t w1)
{
    const uint32_t a = w0 ^ 0x80808080u, b = w1 ^ 0x80808080u;
    return u32x4{bf16_pair((float)(a & 0xFF), (float)((a >> 8) & 0xFF)),
                 bf16_pair((float)((a >> 16) & 0xFF), (float)(a >> 24)),
                 bf16_pair((float)(b & 0xFF), (float)((b >> 8) & 0xFF)),
                 bf16_pair((float)((b >> 16) & 0xFF), (float)(b >> 24))};
}
//   q4: one dword, nibble i (bits 4i..4i+3) = code k_i
__device__ inline u32x4 cvt_q4(uint32_t w)
{
    const uint32_t x = w ^ 0x88888888u;
    const uint32_t lo = x & 0x0F0F0F0Fu;         // k0 k2 k4 k6, one per byte
    const uint32_t hi = (x >> 4) & 0x0F0F0F0Fu;  // k1 k3 k5 k7
    const uint32_t t0 = __builtin_amdgcn_perm(hi, lo, 0x05010400u);  // k0 k1 k2 k3
    const uint32_t t1 = __builtin_amdgcn_perm(hi, lo, 0x07030602u);  // k4 k5 k6 k7
    // each byte u under 0x43: the bf16 pattern 0x4300 | u = 128 + u
    return u32x4{__builtin_amdgcn_perm(0x43434343u, t0, 0x04010400u),
                 __builtin_amdgcn_perm(0x43434343u, t0, 0x04030402u),
                 __builtin_amdgcn_perm(0x43434343u, t1, 0x04010400u),
                 __builtin_amdgcn_perm(0x43434343u, t1, 0x04030402u)};
}

template <int FMT>
struct MidCtx {
    const uint8_t *xb, *cb, *sb;  // wave-uniform bases of the part's first step
    uint32_t xoff[MidGeo<FMT>::XLOADS], coff[MidGeo<FMT>::CLOADS], soff;
    uint8_t *ring, *sring;
    int wave, wm, wn, l32, g;
};

// Issue step s's direct-to-LDS loads into ring slot `stage`, and with SC
// (s % 4 == 0) the scale chunk of steps s .. s + 3.
template <int FMT, bool SC>
__device__ inline void issue(const MidCtx<FMT> &c, uint8_t *stage, int s)
{
    using G = MidGeo<FMT>;
    const uint32_t base = lds_addr(stage);
    const uint8_t *xb = c.xb + s * 128;
    const uint8_t *cb = c.cb + s * G::CROW;
#pragma unroll
    for (int r = 0; r < G::XLOADS; ++r)
        dma16(xb, c.xoff[r], base + (r * THREADS + c.wave * 64) * 16);
#pragma unroll
    for (int r = 0; r < G::CLOADS; ++r)
        dma16(cb, c.coff[r], base + G::XBYTES + (r * THREADS + c.wave * 64) * 16);
    if constexpr (SC)
        dma16(c.sb + (s / SGROUP) * 16, c.soff,
              lds_addr(c.sring + ((s / SGROUP) % SRING) * G::SSLOT) + c.wave * 64 * 16);
}

// Activation fragments of block bl, chunks h = 0, 1, row blocks i = 0, 1.
template <int FMT>
__device__ inline void read_a(const MidCtx<FMT> &c, const uint8_t *stage, int bl, int i,
                              u32x4 (&a)[2])
{
    const int row = c.wm * 64 + i * 32 + c.l32;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        const int lc = 4 * bl + 2 * c.g + h;
        a[h] = *reinterpret_cast<const u32x4 *>(stage + (row * 8 + (lc ^ xswz(row))) * 16);
    }
}

// The lane's codes of block bl for column block j (int8: 16 bytes, q4: 8).
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
template <int FMT>
using Raw = typename std::conditional<FMT == QL_FMT_INT8, u32x4, u32x2>::type;
template <int FMT>
__device__ inline Raw<FMT> read_codes(const MidCtx<FMT> &c, const uint8_t *stage, int bl, int j)
{
    using G = MidGeo<FMT>;
    const int row = c.wn * 64 + j * 32 + c.l32;
    if constexpr (FMT == QL_FMT_INT8)
        return *reinterpret_cast<const u32x4 *>(
            stage + G::XBYTES + (row * G::CCH + ((2 * bl + c.g) ^ cswz<FMT>(row))) * 16);
    else
        return *reinterpret_cast<const u32x2 *>(
            stage + G::XBYTES + (row * G::CCH + (bl ^ cswz<FMT>(row))) * 16 + 8 * c.g);
}

// weight fragment of chunk h from the codes
template <int FMT>
__device__ inline u32x4 convert(const Raw<FMT> &r, int h)
{
    u32x4 v;
    if constexpr (FMT == QL_FMT_INT8)
        v = cvt_int8(r[2 * h], r[2 * h + 1]);
    else
        v = cvt_q4(r[h]);
    pin(v);
    return v;
}

// acc += s * p, the block scale applied to one tile's block partial
__device__ inline void scale_add(f32x16 &acc, float s, const f32x16 &p)
{
#pragma unroll
    for (int r = 0; r < 16; ++r)
        acc[r] = __builtin_fmaf(s, p[r], acc[r]);
    pin(acc);
}

// One block (32 k) of the wavefront's four tiles.  The MFMAs go out in
// groups the compiler may not reorder across; behind each group runs the
// VALU work that does not wait for it: the scale FMAs of the tile before
// (its partial is complete by then), and the reads and conversions of the
// next block's operands.  The last tile's FMAs are left to the caller
// (pend, ps), to run behind the next block's first MFMAs.
//   a, b:   this block's fragments (row blocks i / column blocks j, chunks h)
//   an, bn: the next block's, read here when NEXT (from stage nstage, block
//           nbl)
template <int FMT, bool NEXT>
__device__ inline void block(const MidCtx<FMT> &c, const u32x4 (&a)[2][2], const u32x4 (&b)[2][2],
                             const float (&sc)[2], f32x16 (&acc)[2][2], f32x16 &pend, float &ps,
                             const uint8_t *nstage, int nbl, u32x4 (&an)[2][2], u32x4 (&bn)[2][2])
{
    using G = MidGeo<FMT>;
    const u32x4 offm = {G::OFFW, G::OFFW, G::OFFW, G::OFFW};
    const f32x16 zero = {};
    // offset terms of both row blocks; the previous block's last tile
    f32x16 t0 = mfma(a[0][0], offm, zero);
    t0 = mfma(a[0][1], offm, t0);
    f32x16 t1 = mfma(a[1][0], offm, zero);
    t1 = mfma(a[1][1], offm, t1);
    pin(t0);
    pin(t1);
    scale_add(acc[1][1], ps, pend);
    __builtin_amdgcn_sched_barrier(0);
    // tile (0, 0)
    f32x16 p = mfma(a[0][0], b[0][0], t0);
    p = mfma(a[0][1], b[0][1], p);
    pin(p);
    Raw<FMT> r0, r1;
    if constexpr (NEXT) {
        read_a<FMT>(c, nstage, nbl, 0, an[0]);
        r0 = read_codes<FMT>(c, nstage, nbl, 0);
        pin(an[0][0]), pin(an[0][1]), pin(r0);
    }
    __builtin_amdgcn_sched_barrier(0);
    // tile (0, 1)
    f32x16 q = mfma(a[0][0], b[1][0], t0);
    q = mfma(a[0][1], b[1][1], q);
    pin(q);
    scale_add(acc[0][0], sc[0], p);
    if constexpr (NEXT) {
        read_a<FMT>(c, nstage, nbl, 1, an[1]);
        r1 = read_codes<FMT>(c, nstage, nbl, 1);
        pin(an[1][0]), pin(an[1][1]), pin(r1);
    }
    __builtin_amdgcn_sched_barrier(0);
    // tile (1, 0)
    p = mfma(a[1][0], b[0][0], t1);
    p = mfma(a[1][1], b[0][1], p);
    pin(p);
    scale_add(acc[0][1], sc[1], q);
    if constexpr (NEXT) {
        bn[0][0] = convert<FMT>(r0, 0);
        bn[0][1] = convert<FMT>(r0, 1);
    }
    __builtin_amdgcn_sched_barrier(0);
    // tile (1, 1)
    q = mfma(a[1][0], b[1][0], t1);
    q = mfma(a[1][1], b[1][1], q);
    pin(q);
    scale_add(acc[1][0], sc[0], p);
    if constexpr (NEXT) {
        bn[1][0] = convert<FMT>(r1, 0);
        bn[1][1] = convert<FMT>(r1, 1);
    }
    __builtin_amdgcn_sched_barrier(0);
    pend = q;
    ps = sc[1];
}

// The products of step s (ring slot `stage`): both blocks.  Block 0's
// operands are read first; block 1's behind block 0's MFMAs.
template <int FMT, int U>
__device__ inline void compute(const MidCtx<FMT> &c, const uint8_t *stage, int s,
                               f32x16 (&acc)[2][2], f32x16 &pend, float &ps)
{
    using G = MidGeo<FMT>;
    // scales of the step's two blocks for this lane's weight rows (one
    // dword per column block: block 2 U in the low half, 2 U + 1 in the high)
    float sc[2][2];
#pragma unroll
    for (int j = 0; j < 2; ++j) {
        const int row = c.wn * 64 + j * 32 + c.l32;
        const uint32_t w = *reinterpret_cast<const uint32_t *>(
            c.sring + ((s / SGROUP) % SRING) * G::SSLOT + row * 16 + U * 4);
        sc[0][j] = (float)__builtin_bit_cast(_Float16, (uint16_t)(w & 0xFFFFu));
        sc[1][j] = (float)__builtin_bit_cast(_Float16, (uint16_t)(w >> 16));
    }
    u32x4 a0[2][2], b0[2][2], a1[2][2], b1[2][2];
    read_a<FMT>(c, stage, 0, 0, a0[0]);
    read_a<FMT>(c, stage, 0, 1, a0[1]);
#pragma unroll
    for (int j = 0; j < 2; ++j) {
        const Raw<FMT> r = read_codes<FMT>(c, stage, 0, j);
        b0[j][0] = convert<FMT>(r, 0);
        b0[j][1] = convert<FMT>(r, 1);
    }
    block<FMT, true>(c, a0, b0, sc[0], acc, pend, ps, stage, 1, a1, b1);
    block<FMT, false>(c, a1, b1, sc[1], acc, pend, ps, stage, 0, a0, b0);
}

// Up to four outputs at the right edge of a row, or of a layer whose
// epilogue cannot take groups of four, one at a time.
__device__ inline void store_edge(const Epilogue &ep, float *Y, int64_t idx, int n, int N,
                                  f32x4 v, bool plain)
{
#pragma unroll 1
    for (int e = 0; e < 4 && n + e < N; ++e) {
        if (plain)
            Y[idx + e] = v[e];
        else
            epi_store(ep, Y, idx + e, n + e, v[e]);
    }
}

// Wait until stage s has landed: loads complete in issue order, so it is
// enough that only the y younger stages already issued (s + 1 .. s + y)
// remain in flight, each with LOADS loads per thread plus one for each that
// starts a scale chunk.
template <int FMT, int U, int Y>
__device__ inline void wait_stage(int y)
{
    using G = MidGeo<FMT>;
    if constexpr (Y > 0) {
        if (y == Y) {
            __builtin_amdgcn_s_waitcnt(vmcnt_imm(Y * G::LOADS + (U + Y) / SGROUP));
            return;
        }
        wait_stage<FMT, U, Y - 1>(y);
    } else {
        __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));
    }
}

// Step s = 4 t + U of the part (ns steps, a multiple of 4).
template <int FMT, int U>
__device__ inline void step(const MidCtx<FMT> &c, int s, int ns, f32x16 (&acc)[2][2],
                            f32x16 &pend, float &ps)
{
    using G = MidGeo<FMT>;
    // every LDS read of the previous step has completed; stage s has landed
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    wait_stage<FMT, U, NST - 2>(min(NST - 2, ns - 1 - s));
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");  // no LDS read moves above the barrier
    // the slot of step s - 1 is free: refill it with step s + NST - 1
    if (s + NST - 1 < ns)
        issue<FMT, (U + NST - 1) % SGROUP == 0>(c, c.ring + ((s + NST - 1) % NST) * G::STAGE,
                                                s + NST - 1);
    compute<FMT, U>(c, c.ring + (s % NST) * G::STAGE, s, acc, pend, ps);
}

template <int FMT>
__global__ __launch_bounds__(THREADS, WGS) void qgemm_mid_kernel(const GroupArgs args)
{
    using G = MidGeo<FMT>;
    __shared__ __align__(16) uint8_t ring[G::LDS];

    // layer of workgroup p: every layer spread over all 8 XCDs; within it
    // each XCD takes a contiguous range of (tile, part), parts fastest
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
    const int S = d.ksplit;
    const int tile = local / S, part = local - tile * S;
    const int tm = tile % d.tiles_m, tn = tile / d.tiles_m;
    const int M = d.M, N = d.N, K = d.K, nb = K >> 5;
    const int m0 = tm * BM, n0 = tn * BN;
    const int crow = FMT == QL_FMT_INT8 ? K : K / 2;
    const int tid = threadIdx.x;

    // this part's steps [s0, s0 + ns): psteps % 4 == 0 and K % 256 == 0, so
    // ns is a positive multiple of 4 and s0 starts a scale chunk
    const int s0 = part * d.psteps;
    const int ns = min(K >> 6, s0 + d.psteps) - s0;

    MidCtx<FMT> c;
    c.wave = tid >> 6;
    c.wm = c.wave & 1;
    c.wn = c.wave >> 1;
    c.l32 = tid & 31;
    c.g = (tid >> 5) & 1;
    c.ring = ring;
    c.sring = ring + NST * G::STAGE;
    c.xb = reinterpret_cast<const uint8_t *>(d.X) + (int64_t)m0 * K * 2 + (int64_t)s0 * 128;
    c.cb = d.codes + (int64_t)n0 * crow + (int64_t)s0 * G::CROW;
    c.sb = reinterpret_cast<const uint8_t *>(d.scales) + (int64_t)n0 * nb * 2 +
           (int64_t)(s0 / SGROUP) * 16;
    // activations: slot = row * 8 + (chunk ^ xswz(row)); rows past M repeat
    // the last row (their outputs are never stored)
#pragma unroll
    for (int r = 0; r < G::XLOADS; ++r) {
        const int slot = r * THREADS + tid;
        const int row = slot >> 3;
        const int lc = (slot & 7) ^ xswz(row);
        const int m = min(m0 + row, M - 1) - m0;
        c.xoff[r] = (uint32_t)(m * K * 2 + lc * 16);
    }
    // codes: slot = row * CCH + (chunk ^ cswz(row)); rows past N repeat the
    // last row
#pragma unroll
    for (int r = 0; r < G::CLOADS; ++r) {
        const int slot = r * THREADS + tid;
        const int row = slot / G::CCH;
        const int lc = (slot % G::CCH) ^ cswz<FMT>(row);
        const int n = min(n0 + row, N - 1) - n0;
        c.coff[r] = (uint32_t)(n * crow + lc * 16);
    }
    // scales: thread t fetches the chunk of weight row t % 128
    c.soff = (uint32_t)((min(n0 + (tid & (BN - 1)), N - 1) - n0) * nb * 2);

    // the first NST - 1 stages (those the part has)
    issue<FMT, true>(c, ring, 0);
#pragma unroll
    for (int q = 1; q < NST - 1; ++q)
        if (q < ns) {
            if (q % SGROUP == 0)
                issue<FMT, true>(c, ring + q * G::STAGE, q);
            else
                issue<FMT, false>(c, ring + q * G::STAGE, q);
        }

    f32x16 acc[2][2];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
            acc[i][j] = f32x16{};

    // the last tile's block partial waits for its scale FMAs until behind
    // the next block's first MFMAs (nothing pending before the first block)
    f32x16 pend = {};
    float ps = 0.0f;
#pragma unroll 1
    for (int s = 0; s < ns; s += 4) {
        step<FMT, 0>(c, s, ns, acc, pend, ps);
        step<FMT, 1>(c, s + 1, ns, acc, pend, ps);
        step<FMT, 2>(c, s + 2, ns, acc, pend, ps);
        step<FMT, 3>(c, s + 3, ns, acc, pend, ps);
    }
    scale_add(acc[1][1], ps, pend);

    // Stores.  Register r of tile (i, j) is row wm * 64 + i * 32 + 8 (r / 4)
    // + 4 g + r % 4, column wn * 64 + j * 32 + l32 of the tile.  Each 32 x 32
    // tile goes through a wavefront-private 4 KB LDS patch, written in that
    // layout and read back as rows, so that a lane stores 4 consecutive
    // outputs.  Ring slot ns % NST is free: it held step ns - NST (or no
    // step), which every wavefront finished before the barrier of step
    // ns - NST + 1, and no stage is issued into it after that; a wavefront reads only what it wrote (LDS
    // operations of one wavefront complete in order), so no barrier is
    // needed.  A part of a split layer stores its plain partial output (the
    // sum launch adds the parts in order and applies the epilogue).
    static_assert(4 * 4096 <= G::STAGE, "the patches fit a ring slot");
    float *const patch = reinterpret_cast<float *>(ring + (ns % NST) * G::STAGE) + c.wave * 1024;
    const bool to_part = S > 1;
    float *const Yd = to_part ? d.part + (int64_t)part * M * N : d.Y;
    const bool vec = to_part ? (N & 3) == 0 : epi_vec_ok(d.ep, d.Y, N);
    const int lane = tid & 63;
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) {
#pragma unroll
            for (int r = 0; r < 16; ++r)
                patch[(8 * (r / 4) + 4 * c.g + (r % 4)) * 32 + c.l32] = acc[i][j][r];
            const int n = n0 + c.wn * 64 + j * 32 + 4 * (lane & 7);
#pragma unroll
            for (int t = 0; t < 4; ++t) {
                const int rl = 8 * t + (lane >> 3);
                const f32x4 v = *reinterpret_cast<const f32x4 *>(patch + rl * 32 + 4 * (lane & 7));
                const int m = m0 + c.wm * 64 + i * 32 + rl;
                if (m >= M || n >= N)
                    continue;
                const int64_t idx = (int64_t)m * N + n;
                if (vec && n + 3 < N) {
                    if (to_part)
                        *reinterpret_cast<f32x4 *>(Yd + idx) = v;
                    else
                        epi_store4(d.ep, Yd, idx, n, v, false);
                } else {
                    store_edge(d.ep, Yd, idx, n, N, v, to_part);
                }
            }
        }
}

}  // namespace

int mid_tile_bm() { return BM; }
int mid_tile_bn() { return BN; }
int mid_wgs_per_cu() { return WGS; }

hipError_t launch_qgemm_mid(int fmt, const GroupArgs &args, hipStream_t stream)
{
    dim3 grid((unsigned)args.total_tiles), block(THREADS);
    if (fmt == QL_FMT_INT8)
        hipLaunchKernelGGL(qgemm_mid_kernel<QL_FMT_INT8>, grid, block, 0, stream, args);
    else if (fmt == QL_FMT_Q4)
        hipLaunchKernelGGL(qgemm_mid_kernel<QL_FMT_Q4>, grid, block, 0, stream, args);
    else
        return hipErrorInvalidValue;
    return hipGetLastError();
}

}  // namespace qlk
