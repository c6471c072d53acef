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
// with the whole K (or one K part of a split reduction) accumulated in fp32
// by v_mfma_f32_32x32x16_f16.  f[n] is chosen per weight row (and K part)
// from the largest scale of the row's blocks in the part, so that every
// |W'| is below 2^15: c is made exact in fp16 by a magic-number add (the fp16 bit
// pattern 0x6400 | u is 1024 + u) and one packed fp16 multiply by the scaled
// scale rounds c * s to 11 significant bits.  No per-block work remains on
// the accumulators, which is what made the exact per-block form
// (qgemm.hip: an fp32 FMA per output element per block) bound by VALU issue.
//
// Matrix instruction.  On gfx950 the 32 x 32 x 16 fp16 MFMA sustains about
// twice the flop rate of the 16 x 16 x 32 one (each takes the same issue
// time, the larger one does twice the work), so the tile is built from it.
// Its operand layout: lane l holds A[l % 32][8 (l / 32) + e] and
// B[8 (l / 32) + e][l % 32] for e = 0..7, and accumulator register r of lane
// l is D[8 (r / 4) + 4 (l / 32) + r % 4][l % 32].
//
// k order.  The sum over k does not care which k a given MFMA slot holds, as
// long as A and B agree.  Within a 64-k step, slot e of lane group g = l / 32
// in the step's 16-k chunk q holds k = 32 g + 8 q + e (int8), or
// 32 g + 8 q + Q4_SLOT[e] (q4: the order in which the code conversion
// produces an 8-k group; the activation copy is stored in that order).  Then
// every lane's k over the whole step is one contiguous run of 32 = one scale
// block: its weight codes for the step are one 16-byte (q4) or 32-byte
// (int8) LDS read, it needs one scale per weight row per step, and each
// activation fragment is one 16-byte chunk of the row.
//
// Tile: 256 threads (4 wavefronts) compute BM x BN = 128 x 256 of Y.  Each
// wavefront owns a 128 x 64 strip (4 x 2 MFMA tiles of 32 x 32): every
// dequantized weight fragment feeds 4 MFMAs and every activation fragment 2.
// The wide N extent halves the activation traffic per flop against a square
// tile: the fp16 activations (2 bytes per element, re-read once per column
// tile) are the larger operand stream next to 4-bit codes.
//
// Memory pipeline: activations, codes and scales move from global memory to
// LDS with the gfx950 direct-to-LDS loads (no VGPRs, no VALU), through a ring
// of NST stages of 64 k each (two scale blocks).  The step barrier sits
// before the last 16-k chunk of a step: by then every wavefront has read
// all of the step's slot, so that slot is refilled at once (with the step
// NST ahead), and the last chunk's MFMAs run while the next step's first
// operands are read and converted (no stall between steps).  Each lane's
// offset within the tile is
// computed once; per step only the wave-uniform base (an SGPR pair)
// advances.  The loads are issued from inline asm so that the compiler's
// wait insertion, which cannot tell the ring stages apart and would drain
// every load in flight before each LDS read, stays out of the way: the
// kernel waits for each stage explicitly (s_waitcnt vmcnt, then s_barrier; a
// __syncthreads() would also drain the ring).  Nothing else here uses M0.
//
// LDS layouts are XOR-swizzled at 16-byte granularity so that the fragment
// reads of 8 (32 banks) or 16 (64 banks) consecutive lanes hit distinct
// banks.  A direct-to-LDS load writes lane t's data to slot base + t, so the
// swizzle is applied by choosing which global chunk each lane fetches.
//
// fp16 weights (QL_FMT_F16, the unquantized reference format) go through the
// same kernel: the weight words are the MFMA operand as they are (no
// conversion, f = 0, no scales), 128 bytes per row per stage, one workgroup
// per CU.
//
// Tile order: within a layer, groups of 4 row tiles walked row-tile fastest;
// each of the 8 XCDs takes a contiguous range of one layer's tiles (L2
// reuse), and every layer of a grouped launch is spread over all XCDs.  Long
// reductions may be cut into K parts (ksplit, see the split reduction at the
// end of the kernel).
#include <algorithm>

#include "epilogue.h"
#include "internal.h"

namespace qlk {
namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef _Float16 half2v __attribute__((ext_vector_type(2)));

// Tile shape (compile-time): each of WAVES wavefronts owns MSUB x NSUB MFMA
// tiles of 32 x 32.  The shipped shape is MSUB = 4, NSUB = 2, WAVES = 4:
// 128 x 256 tiles, two workgroups per CU.  Shapes with 256 accumulators per
// lane (MSUB * NSUB = 16: one workgroup, one wavefront per SIMD) or 8
// wavefronts build too; measured on the q4 step they were slower.
#ifndef QL_WIDE_MSUB
#define QL_WIDE_MSUB 4
#endif
#ifndef QL_WIDE_WAVES
#define QL_WIDE_WAVES 4
#endif
constexpr int WAVES = QL_WIDE_WAVES, THREADS = 64 * WAVES;
#ifndef QL_WIDE_NSUB
#define QL_WIDE_NSUB 2
#endif
constexpr int MSUB = QL_WIDE_MSUB, NSUB = QL_WIDE_NSUB, BM = 32 * MSUB, BN = WAVES * 32 * NSUB;
constexpr int WN = 32 * NSUB;  // columns per wavefront
constexpr int GROUP_M = 4;
constexpr int WGS_PER_CU = MSUB * NSUB > 8 || WAVES == 8 ? 1 : 2;
// fp16 weights (the unquantized reference format) take 128 bytes per row per
// stage: one workgroup per CU
template <int FMT>
constexpr int wgs_per_cu() { return FMT == QL_FMT_F16 ? 1 : WGS_PER_CU; }
constexpr int MAXSPLIT = 4;  // parts per output tile (split reduction)

template <int FMT>
struct Geo {
    static constexpr int XBYTES = BM * 64 * 2;                 // activations per stage
    static constexpr int CROW = FMT == QL_FMT_INT8 ? 64 : FMT == QL_FMT_Q4 ? 32 : 128;  // weight
                                                               // bytes per row per stage
    static constexpr int CCH = CROW / 16;                      // 16-byte chunks per code row
    static constexpr int CBYTES = BN * CROW;
    static constexpr int STAGE = XBYTES + CBYTES;
    // scales travel apart: one 16-byte chunk (8 blocks = 4 steps) per weight
    // row every 4 steps, into a 2-slot ring; a per-step load would cost one
    // memory request per row for 4 bytes
    static constexpr int SGROUP = 4, SSLOT = FMT == QL_FMT_F16 ? 0 : BN * 16;
    // ring depth: three stages where the LDS budget of the resident
    // workgroups allows them, else two
    static constexpr int NST = wgs_per_cu<FMT>() * (3 * STAGE + 2 * SSLOT) <= 160 * 1024 ? 3 : 2;
    static constexpr int XLOADS = XBYTES / 16 / THREADS;
    static constexpr int CLOADS = CBYTES / 16 / THREADS;
    static constexpr int SPT = FMT == QL_FMT_F16 ? 0 : BN / THREADS;  // scale chunks per
                                                                     // thread per group
    static constexpr int LOADS = XLOADS + CLOADS;  // direct-to-LDS loads per step (+SPT every 4)
    static constexpr int LDS = NST * STAGE + 2 * SSLOT;
    static_assert(XBYTES % (16 * THREADS) == 0 && CBYTES % (16 * THREADS) == 0,
                  "every thread issues the same number of 16-byte loads per stage");
    static_assert(BN % THREADS == 0, "whole scale chunks per thread");
    static_assert(wgs_per_cu<FMT>() * LDS <= 160 * 1024, "resident workgroups per CU");
};

__device__ inline constexpr int vmcnt_imm(int v)
{
    // gfx9 s_waitcnt encoding: vmcnt[3:0] + vmcnt[5:4] at bits 15:14;
    // expcnt (bits 6:4) and lgkmcnt (bits 11:8) left at "no wait"
    return (v & 15) | (((v >> 4) & 3) << 14) | (7 << 4) | (15 << 8);
}

// 16-byte chunk swizzles (physical chunk = logical ^ swz(row)); each keeps
// the reads described above free of bank conflicts for 32 or 64 banks
__device__ inline int xswz(int row) { return (row & 7) ^ ((row >> 3) & 1); }
template <int FMT>
__device__ inline int cswz(int row)
{
    if constexpr (FMT == QL_FMT_F16)
        return xswz(row);  // 8 chunks per row, as the activations
    return FMT == QL_FMT_INT8 ? ((row >> 1) ^ (row >> 3)) & 3 : ((row >> 2) ^ (row >> 3)) & 1;
}

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

__device__ inline f32x16 mfma32(u32x4 a, u32x4 b, f32x16 c)
{
    return __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(half8, a),
                                                  __builtin_bit_cast(half8, b), c, 0, 0, 0);
}

__device__ inline uint32_t h2mul_add(uint32_t v, half2v bias, half2v sp)
{
    // (v + bias) is exact (an fp16 integer), then one rounded multiply
    return __builtin_bit_cast(uint32_t, (__builtin_bit_cast(half2v, v) + bias) * sp);
}

// 16-byte store / load at device coherence (write-through to, and read
// from, the level shared by all XCDs).  A store of more than 8 bytes keeps
// reading its data registers for a cycle after issue; the compiler's hazard
// check does not look inside inline asm, so the wait state that keeps the
// next VALU write from those registers back is part of the statement.
__device__ inline void st_coherent(float *p, f32x4 v)
{
    asm volatile("global_store_dwordx4 %0, %1, off sc1\n\ts_nop 1" : : "v"(p), "v"(v) : "memory");
}

__device__ inline f32x4 ld_coherent(const float *p)
{
    // agent-scope atomic loads: sc1, and waited for by the compiler (a load
    // from inline asm would not be: the compiler could reuse its destination
    // registers before the data arrives)
    const uint32_t *q = reinterpret_cast<const uint32_t *>(p);
    f32x4 v;
#pragma unroll
    for (int k = 0; k < 4; ++k)
        v[k] = __uint_as_float(__hip_atomic_load(q + k, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
    return v;
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
    uint32_t xoff[Geo<FMT>::XLOADS], coff[Geo<FMT>::CLOADS], soff[Geo<FMT>::SPT];
    uint8_t *sring;  // the scale ring (2 slots of BN rows x 16 bytes)
    int wave, l32, g;
    int f[NSUB];  // weight row (wave * WN + j * 32 + l32) enters as W * 2^f[j]
};

// Issue the direct-to-LDS loads of step s into one ring stage, and with
// SCALES (s % 4 == 0) the scales of steps s .. s + 3 into their ring slot.
template <int FMT, bool SCALES>
__device__ inline void issue_stage(const Ctx<FMT> &c, uint8_t *stage, int s)
{
    using G = Geo<FMT>;
    const uint32_t base = lds_addr(stage);
    const uint8_t *xb = c.xbase + s * 128;  // 64 fp16 per row per step
    const uint8_t *cb = c.cbase + s * G::CROW;
#pragma unroll
    for (int r = 0; r < G::XLOADS; ++r)
        dma16(xb, c.xoff[r], base + (r * THREADS + c.wave * 64) * 16);
#pragma unroll
    for (int r = 0; r < G::CLOADS; ++r)
        dma16(cb, c.coff[r], base + G::XBYTES + (r * THREADS + c.wave * 64) * 16);
    if constexpr (SCALES) {
        const int g = s / G::SGROUP;
#pragma unroll
        for (int h = 0; h < G::SPT; ++h)
            dma16(c.sbase + g * 16, c.soff[h],
                  lds_addr(c.sring + (g & 1) * G::SSLOT) + (h * THREADS + c.wave * 64) * 16);
    }
}

// fp16 pair {s * 2^f, s * 2^f} for the scale bits b
__device__ inline half2v scaled_pair(uint32_t b, int f)
{
    const _Float16 s = __builtin_amdgcn_ldexph(__builtin_bit_cast(_Float16, (uint16_t)b), f);
    return half2v{s, s};
}

// Word w (two fp16 weights) of weight fragment (chunk q) from the lane's raw
// codes of the step, one word at a time so that the conversion can be
// spread between MFMAs.  c is placed under the fp16 exponent pattern 0x64
// as an unsigned byte u (0x6400 | u = 1024 + u) by a v_perm whose other
// source is 0x64646464, then (1024 + u + bias) is exact and one packed
// multiply by s' rounds.
//   int8: u = c + 128 (byte ^ 0x80), bias -1152; the 8 k of a word pair in
//         natural order.
//   q4:   u = c + 8 (nibble ^ 8), low nibbles (even k) and high nibbles (odd
//         k) separated into bytes first, bias -1032.  A v_perm takes two
//         bytes of one source, so the words hold (k0, k2), (k4, k6),
//         (k1, k3), (k5, k7) of each 8-k group: slot e holds k = Q4_SLOT[e],
//         and the activations are stored in the same order (xprep.hip).
template <int FMT>
__device__ inline uint32_t deq_word(const uint32_t *raw, int q, int w, half2v sp)
{
    if constexpr (FMT == QL_FMT_F16) {
        return raw[4 * q + w];  // the weights themselves, natural k order
    } else if constexpr (FMT == QL_FMT_INT8) {
        const uint32_t x = raw[2 * q + (w >> 1)] ^ 0x80808080u;
        const half2v bias = {(_Float16)-1152.0f, (_Float16)-1152.0f};
        return h2mul_add(__builtin_amdgcn_perm(0x64646464u, x, (w & 1) ? 0x04030402u : 0x04010400u),
                         bias, sp);
    } else {
        const uint32_t c = w < 2 ? raw[q] : raw[q] >> 4;
        const uint32_t u = (c & 0x0F0F0F0Fu) ^ 0x08080808u;  // one v_bitop3
        const half2v bias = {(_Float16)-1032.0f, (_Float16)-1032.0f};
        return h2mul_add(__builtin_amdgcn_perm(0x64646464u, u, (w & 1) ? 0x04030402u : 0x04010400u),
                         bias, sp);
    }
}

// An empty statement that the compiler keeps in order with the scheduling
// barriers: a value passed through it is computed in the MFMA group it is
// written in.  (Without it, the optimizer sinks a chunk's weight words
// below its last MFMA, next to the vector they are assembled into, and the
// VALU work that should overlap the MFMAs runs in one block after them.)
__device__ inline uint32_t pin(uint32_t v)
{
    asm volatile("" : "+v"(v));
    return v;
}

// Operands carried from one 16-k chunk to the next, and across the step
// boundary: the step's raw codes and scale pairs (one 32-k block per lane
// and weight fragment j), and the activation and dequantized weight
// fragments of the chunk about to be multiplied.
template <int FMT>
struct Ops {
    uint32_t raw[NSUB][Geo<FMT>::CCH / 2 * 4];
    half2v sp[NSUB];
    u32x4 a[MSUB], B[NSUB];
};

// scale bits of step s (block 2s + g) for this lane's row of fragment j:
// half g of dword s % 4 of the row's chunk, ring slot (s / 4) & 1
template <int FMT>
__device__ inline uint32_t scale_bits(const Ctx<FMT> &c, int s, int j)
{
    using G = Geo<FMT>;
    const int row = c.wave * WN + j * 32 + c.l32;
    return *reinterpret_cast<const uint16_t *>(c.sring + ((s / G::SGROUP) & 1) * G::SSLOT +
                                               row * 16 + (s % G::SGROUP) * 4 + c.g * 2);
}

// the lane's codes of one step for fragment j (its 32-k block)
template <int FMT>
__device__ inline void read_codes(const Ctx<FMT> &c, const uint8_t *stage, int j,
                                  uint32_t (&raw)[Geo<FMT>::CCH / 2 * 4])
{
    using G = Geo<FMT>;
    const int row = c.wave * WN + j * 32 + c.l32;
#pragma unroll
    for (int h = 0; h < G::CCH / 2; ++h) {
        const int lc = c.g * (G::CCH / 2) + h;
        const u32x4 v = *reinterpret_cast<const u32x4 *>(
            stage + G::XBYTES + (row * G::CCH + (lc ^ cswz<FMT>(row))) * 16);
#pragma unroll
        for (int w = 0; w < 4; ++w)
            raw[h * 4 + w] = v[w];
    }
}

// activation fragment of chunk q for row block i
template <int FMT>
__device__ inline u32x4 read_a(const Ctx<FMT> &c, const uint8_t *stage, int q, int i)
{
    const int row = i * 32 + c.l32;
    const int lc = c.g * 4 + q;
    return *reinterpret_cast<const u32x4 *>(stage + (row * 8 + (lc ^ xswz(row))) * 16);
}

// Operands of chunk 0 of a step, from scratch (the first step of a tile).
template <int FMT>
__device__ inline void first_chunk(const Ctx<FMT> &c, const uint8_t *stage, int s, Ops<FMT> &op)
{
#pragma unroll
    for (int j = 0; j < NSUB; ++j) {
        if constexpr (FMT != QL_FMT_F16)
            op.sp[j] = scaled_pair(scale_bits<FMT>(c, s, j), c.f[j]);
        read_codes<FMT>(c, stage, j, op.raw[j]);
    }
#pragma unroll
    for (int i = 0; i < MSUB; ++i)
        op.a[i] = read_a<FMT>(c, stage, 0, i);
#pragma unroll
    for (int j = 0; j < NSUB; ++j)
#pragma unroll
        for (int w = 0; w < 4; ++w)
            op.B[j][w] = deq_word<FMT>(op.raw[j], 0, w, op.sp[j]);
}

// The MSUB x NSUB MFMAs of chunk Q of a step.  Behind each MFMA, in a group
// the compiler may not reorder, goes a share of the next chunk's operand
// preparation, so that the matrix core runs while the VALU and LDS work:
//   Q < 3: the activation fragments (from cur) and weight words of chunk
//          Q + 1, one word per MFMA, one fragment read every NSUB MFMAs;
//   Q = 3 with NEXT: chunk 0 of the next step, from that step's ring slot
//          nxt: its codes and scales (all read behind the first MFMA), its
//          activation fragments, its scale pairs, then its weight words.
// With the last chunk of a step preparing the next step's first one, a
// wavefront goes from the step barrier straight into MFMAs.
template <int FMT, int Q, bool NEXT>
__device__ inline void chunk(const Ctx<FMT> &c, const uint8_t *cur, const uint8_t *nxt, int s,
                             Ops<FMT> &op, f32x16 (&acc)[MSUB][NSUB])
{
    constexpr int KK = MSUB * NSUB, W = 4 * NSUB;
    static_assert(KK >= 4, "the next step's words start behind the fourth MFMA");
    u32x4 an[MSUB], Bn[NSUB];
    uint32_t sb[NSUB];
#pragma unroll
    for (int k = 0; k < KK; ++k) {
        const int i = k / NSUB, j = k % NSUB;
        acc[i][j] = mfma32(op.a[i], op.B[j], acc[i][j]);
        if constexpr (Q < 3) {
            if (k % NSUB == 0)
                an[k / NSUB] = read_a<FMT>(c, cur, Q + 1, k / NSUB);
            if ((k + 1) * 4 % MSUB == 0) {
                const int wd = (k + 1) * 4 / MSUB - 1, jn = wd / 4, w = wd % 4;
                Bn[jn][w] = pin(deq_word<FMT>(op.raw[jn], Q + 1, w, op.sp[jn]));
            }
        } else if constexpr (NEXT) {
            // this step's codes and scale pairs are dead once chunk 3's
            // weight words exist: the next step's take their registers
            if (k == 0) {
#pragma unroll
                for (int jj = 0; jj < NSUB; ++jj) {
                    if constexpr (FMT != QL_FMT_F16)
                        sb[jj] = scale_bits<FMT>(c, s + 1, jj);
                    read_codes<FMT>(c, nxt, jj, op.raw[jj]);
                }
            }
            if (k % NSUB == 0)
                an[k / NSUB] = read_a<FMT>(c, nxt, 0, k / NSUB);
            if constexpr (FMT != QL_FMT_F16) {
                if (k == 2)
#pragma unroll
                    for (int jj = 0; jj < NSUB; ++jj)
                        op.sp[jj] = scaled_pair(sb[jj], c.f[jj]);
            }
            if (k >= 3) {
#pragma unroll
                for (int wd = (k - 3) * W / (KK - 3); wd < (k - 2) * W / (KK - 3); ++wd)
                    Bn[wd / 4][wd % 4] =
                        pin(deq_word<FMT>(op.raw[wd / 4], 0, wd % 4, op.sp[wd / 4]));
            }
        }
        __builtin_amdgcn_sched_barrier(0);
    }
    if constexpr (Q < 3 || NEXT) {
#pragma unroll
        for (int i = 0; i < MSUB; ++i)
            op.a[i] = an[i];
#pragma unroll
        for (int j = 0; j < NSUB; ++j)
            op.B[j] = Bn[j];
    }
}

// One step s = 4 t + U of a tile's main loop (ns steps, a multiple of 4).
// TAIL: s is one of the last 4 steps (s = ns - 4 + U), where whether a
// younger stage is in flight and whether a stage is issued depend on U.
// Every condition is a compile-time one, so the step is one basic block
// and no operand preparation can be moved across the barrier.
// Chunks 0-2 prepare their successors from the step's slot; then every
// wavefront's reads of the slot are complete (lgkmcnt), stage s + 1 has
// landed (loads complete in issue order: only the younger stage s + 2 may
// still be in flight), the barrier, the slot is refilled with step s + NST,
// and chunk 3 runs while step s + 1's chunk 0 is prepared.
template <int FMT, int U, bool TAIL>
__device__ inline void step(const Ctx<FMT> &c, uint8_t *ring, int s, int &slot, Ops<FMT> &op,
                            f32x16 (&acc)[MSUB][NSUB])
{
    using G = Geo<FMT>;
    constexpr int NST = G::NST;
    constexpr bool LAST = TAIL && U == 3;             // s = ns - 1
    constexpr bool ISSUE = !TAIL || U + NST < 4;      // s + NST < ns
    constexpr bool YOUNGER = NST == 3 && (!TAIL || U < 2);  // s + 2 < ns: in flight
    const uint8_t *const cur = ring + slot * G::STAGE;
    const int nslot = slot + 1 == NST ? 0 : slot + 1;
    const uint8_t *const nxt = ring + nslot * G::STAGE;
    chunk<FMT, 0, false>(c, cur, nxt, s, op, acc);
    chunk<FMT, 1, false>(c, cur, nxt, s, op, acc);
    chunk<FMT, 2, false>(c, cur, nxt, s, op, acc);
    if constexpr (!LAST) {
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
        if constexpr (YOUNGER)
            __builtin_amdgcn_s_waitcnt(
                vmcnt_imm(G::LOADS + ((U + 2) % G::SGROUP == 0 ? G::SPT : 0)));
        else
            __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));
        __builtin_amdgcn_s_barrier();
        if constexpr (ISSUE)
            issue_stage<FMT, (U + NST) % G::SGROUP == 0>(c, ring + slot * G::STAGE, s + NST);
        chunk<FMT, 3, true>(c, cur, nxt, s, op, acc);
    } else {
        chunk<FMT, 3, false>(c, cur, nxt, s, op, acc);
    }
    slot = nslot;
}

// EPI: some layer of the launch has an epilogue (bias, GELU, residual or
// bf16 outputs); the kernel without one keeps the plain fp32 store code only
template <int FMT, bool EPI>
__global__ __launch_bounds__(THREADS, wgs_per_cu<FMT>()) void qgemm_wide_kernel(const GroupArgs args)
{
    using G = Geo<FMT>;
    constexpr int NST = G::NST;
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
    const int crow_bytes = FMT == QL_FMT_INT8 ? K : FMT == QL_FMT_Q4 ? K / 2 : 2 * K;

    Ctx<FMT> c;
    c.wave = tid >> 6;
    c.l32 = tid & 31;
    c.g = (tid & 63) >> 5;
    c.xbase = reinterpret_cast<const uint8_t *>(d.X) + (int64_t)m0 * K * 2;
    c.cbase = d.codes + (int64_t)n0 * crow_bytes;
    c.sbase = reinterpret_cast<const uint8_t *>(d.scales) + (int64_t)n0 * nb * 2;
    // activations: stage slot = row * 8 + (chunk ^ xswz(row)); rows past M
    // repeat the last row (their outputs are never stored)
#pragma unroll
    for (int r = 0; r < G::XLOADS; ++r) {
        const int slot = r * THREADS + tid;
        const int row = slot >> 3;
        const int lc = (slot & 7) ^ xswz(row);
        const int m = min(m0 + row, M - 1) - m0;
        c.xoff[r] = (uint32_t)(m * K * 2 + lc * 16);
    }
    // codes: stage slot = row * CCH + (chunk ^ cswz(row)); rows past N
    // repeat the last row
#pragma unroll
    for (int r = 0; r < G::CLOADS; ++r) {
        const int slot = r * THREADS + tid;
        const int row = slot / G::CCH;
        const int lc = (slot % G::CCH) ^ cswz<FMT>(row);
        const int n = min(n0 + row, N - 1) - n0;
        c.coff[r] = (uint32_t)(n * crow_bytes + lc * 16);
    }
    // scales: one 16-byte chunk of weight rows h * THREADS + tid per 4 steps
#pragma unroll
    for (int h = 0; h < G::SPT; ++h)
        c.soff[h] = (uint32_t)((min(n0 + h * THREADS + tid, N - 1) - n0) * nb * 2);
    c.sring = ring + NST * G::STAGE;

    // this part's steps of 64 k: [s0, s0 + ns); s0 is a multiple of the
    // scale group (psteps % 4 == 0, checked by the host)
    const int s0 = part * d.psteps;
    const int ns = min(nb >> 1, s0 + d.psteps) - s0;
    c.xbase += s0 * 128;
    c.cbase += s0 * G::CROW;
    c.sbase += s0 / G::SGROUP * 16;
    // The shifts of the tile's 256 weight rows in this K part (set by the
    // pre-pass from the largest scale of the part's blocks of each row; each
    // part's partial outputs are scaled back exactly before they are stored
    // or added up, so parts may differ): one direct-to-LDS load by wavefront
    // 0, 16 bytes (4 rows) per lane, into the first KB of the scale ring's
    // second slot (filled from step 4 on, after the shifts are read), issued
    // before stage 0 so that the stage 0 wait covers it.
    static_assert(FMT == QL_FMT_F16 || BN * 4 == 64 * 16, "one 16-byte load per lane of a wavefront");
    if constexpr (FMT != QL_FMT_F16)
        if (c.wave == 0)
            dma16(d.wshift + (int64_t)part * d.wsld + n0, (uint32_t)(tid & 63) * 16,
                  lds_addr(c.sring + G::SSLOT));
    // ns >= 4 > NST: every ring slot gets its first stage
    issue_stage<FMT, true>(c, ring, 0);
#pragma unroll
    for (int q = 1; q < NST; ++q)
        issue_stage<FMT, false>(c, ring + q * G::STAGE, q);

    f32x16 acc[MSUB][NSUB];
#pragma unroll
    for (int i = 0; i < MSUB; ++i)
#pragma unroll
        for (int j = 0; j < NSUB; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r)
                acc[i][j][r] = 0.f;

    // Stage waits: loads complete in issue order, so waiting until only the
    // loads of the younger stages already issued remain outstanding means
    // all of a stage has landed.  A stage starting a scale group carries one
    // more load per thread.  The first wait leaves stages 1 .. NST - 1 in
    // flight (ns >= 4 > NST - 1: K parts are whole scale groups); the
    // shifts, issued before stage 0, have landed with it.
    static_assert(NST == 2 || NST == 3, "wait counts cover at most one younger stage");
    __builtin_amdgcn_s_waitcnt(vmcnt_imm((NST - 1) * G::LOADS));
    __builtin_amdgcn_s_barrier();
#pragma unroll
    for (int j = 0; j < NSUB; ++j)  // (fp16 weights enter as they are)
        c.f[j] = FMT == QL_FMT_F16 ? 0
                                   : reinterpret_cast<const int *>(
                                         c.sring + G::SSLOT)[c.wave * WN + j * 32 + c.l32];
    Ops<FMT> op;
    first_chunk<FMT>(c, ring, 0, op);
    // The main loop runs at a raised wave priority: with two workgroups on
    // a CU, the one in its main loop is issued ahead of the other's prologue
    // and epilogue (measured on the q4 step block call: 219.4 -> 216.8 us
    // against raising it for the MFMAs only).
    int slot = 0;
    __builtin_amdgcn_s_setprio(1);
#pragma unroll 1
    for (int s = 0; s + 4 < ns; s += 4) {
        step<FMT, 0, false>(c, ring, s, slot, op, acc);
        step<FMT, 1, false>(c, ring, s + 1, slot, op, acc);
        step<FMT, 2, false>(c, ring, s + 2, slot, op, acc);
        step<FMT, 3, false>(c, ring, s + 3, slot, op, acc);
    }
    step<FMT, 0, true>(c, ring, ns - 4, slot, op, acc);
    step<FMT, 1, true>(c, ring, ns - 3, slot, op, acc);
    step<FMT, 2, true>(c, ring, ns - 2, slot, op, acc);
    step<FMT, 3, true>(c, ring, ns - 1, slot, op, acc);
    __builtin_amdgcn_s_setprio(0);

    // Epilogue.  Register r of tile (i, j) is row i * 32 + 8 (r / 4) + 4 g +
    // r % 4, column wave * WN + j * 32 + l32 of the tile; it returns to the
    // scale of X * W^T by the exact factor 2^(e[m] - f[n]).  Values are taken
    // from the accumulators as they are stored (no second copy of the tile
    // in registers).
    // Ring slot ns % NST is free now: it held step ns - NST, which every
    // wavefront read before an earlier step barrier, and no stage is issued
    // into it after that.  Each wavefront keeps its own copy of the tile's
    // row shifts there (no barrier: a wavefront reads only what it wrote,
    // and LDS operations of one wavefront complete in order), read back 4
    // consecutive rows per 16-byte read; rows past M repeat the last row
    // (their outputs are never stored).
    uint8_t *const spare = ring + (ns % NST) * G::STAGE;
    static_assert(WAVES * 4096 + WAVES * BM * 4 <= G::STAGE, "patches and row shifts fit a slot");
    int *const rowexp = reinterpret_cast<int *>(spare + WAVES * 4096) + c.wave * BM;
    for (int t = tid & 63; t < BM; t += 64)
        rowexp[t] = d.xexp[min(m0 + t, M - 1)];
    auto shifts = [&](int i, int (&ex)[16]) {
#pragma unroll
        for (int b = 0; b < 4; ++b) {
            const int4 v = *reinterpret_cast<const int4 *>(rowexp + i * 32 + 8 * b + 4 * c.g);
            ex[4 * b] = v.x;
            ex[4 * b + 1] = v.y;
            ex[4 * b + 2] = v.z;
            ex[4 * b + 3] = v.w;
        }
    };
    auto group = [&](int i, int j, int h, const int (&ex)[16]) {
        return f32x4{__builtin_amdgcn_ldexpf(acc[i][j][4 * h], ex[4 * h] - c.f[j]),
                     __builtin_amdgcn_ldexpf(acc[i][j][4 * h + 1], ex[4 * h + 1] - c.f[j]),
                     __builtin_amdgcn_ldexpf(acc[i][j][4 * h + 2], ex[4 * h + 2] - c.f[j]),
                     __builtin_amdgcn_ldexpf(acc[i][j][4 * h + 3], ex[4 * h + 3] - c.f[j])};
    };
    // Y stores: each 32 x 32 tile (the four groups h of (i, j)) goes through
    // a wavefront-private 4 KB LDS patch, written in the MFMA layout and
    // read back as rows, so that every lane stores 16 contiguous bytes and
    // each store instruction covers 8 whole 128-byte row segments (the
    // register layout would give 4-byte stores).  A wavefront reads only
    // what it wrote, in order, so no barrier is needed.  The patches live
    // in the free ring slot too.
    float *const patch = reinterpret_cast<float *>(spare) + c.wave * 1024;
    // destination: Y, or this part's plain partial output when the parts
    // are summed by a separate launch (split_sum_kernel)
    const bool to_part = (S > 1 && !d.cnt) || d.part_out;
    float *const Yd = to_part ? d.part + (int64_t)part * M * N : d.Y;
    const bool vec = (N & 3) == 0 && ((uintptr_t)Yd & 15) == 0;
    // a layer epilogue beyond the plain fp32 store (final outputs only)
    const bool epi = EPI && !to_part && epi_active(d.ep);
    // the per-column epilogue operands (bias, steering term) of this lane's
    // column groups, loaded once before the first store: a load issued after
    // stores waits for them too (the vector memory counter retires in order)
    f32x4 bcol[NSUB], scol[NSUB];
    float alpha = 0.0f;
#pragma unroll
    for (int j = 0; j < NSUB; ++j) {
        bcol[j] = f32x4{0.f, 0.f, 0.f, 0.f};
        scol[j] = bcol[j];
    }
    if (epi) {
#pragma unroll
        for (int j = 0; j < NSUB; ++j) {
            const int n = n0 + c.wave * WN + j * 32 + 4 * (tid & 7);
            if (n < N) {
                if (d.ep.bias)
                    bcol[j] = *reinterpret_cast<const f32x4 *>(d.ep.bias + n);
                scol[j] = epi_steer4<f32x4>(d.ep, n, alpha);
            }
        }
    }
    auto store_tile = [&](int i, int j, const f32x4 (&y)[4]) {
        const int lane = tid & 63;
        const int cq = lane & 7;          // 4-column group of the row
        const int n = n0 + c.wave * WN + j * 32 + 4 * cq;
        if (!epi) {
#pragma unroll
            for (int h = 0; h < 4; ++h)
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    patch[(8 * h + 4 * c.g + e) * 32 + c.l32] = y[h][e];
#pragma unroll
            for (int t = 0; t < 4; ++t) {
                const int rl = 8 * t + (lane >> 3);  // row within the 32-row tile
                const f32x4 v = *reinterpret_cast<const f32x4 *>(patch + rl * 32 + 4 * cq);
                const int m = m0 + i * 32 + rl;
                if (m >= M)
                    continue;
                float *const dst = Yd + (int64_t)m * N + n;
                if (n + 3 < N && vec) {
                    // streaming store for Y (not read again here: letting it
                    // allocate would evict the activation and code lines that
                    // other tiles still re-read); partials, which the sum
                    // launch reads next, stay cacheable
                    if (to_part)
                        *reinterpret_cast<f32x4 *>(dst) = v;
                    else
                        __builtin_nontemporal_store(v, reinterpret_cast<f32x4 *>(dst));
                } else {
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        if (n + e < N)
                            dst[e] = v[e];
                }
            }
            return;
        }
        // with the epilogue: the four rows' residual loads go out first
        // (before the patch round trip, which hides part of their latency),
        // without allocating in the caches (each row is read once; the
        // activation and code lines that other tiles re-read stay).  The
        // layer takes groups of four (the host routes any other layer with an
        // epilogue through plain partials and the sum launch), so this is
        // straight-line code with predicated stores.
        const int mb = m0 + i * 32 + (lane >> 3);  // row of iteration 0
        // groups of four (N % 4 == 0: a lane's group is whole or beyond N)
        const bool col_ok = n < N;
        const f32x4 b4 = bcol[j], s4 = scol[j];
        f32x4 r[4] = {b4, b4, b4, b4};
        if (d.ep.resid) {
#pragma unroll
            for (int t = 0; t < 4; ++t)
                if (col_ok && mb + 8 * t < M)
                    r[t] = __builtin_nontemporal_load(reinterpret_cast<const f32x4 *>(
                        d.ep.resid + (int64_t)(mb + 8 * t) * N + n));
        }
#pragma unroll
        for (int h = 0; h < 4; ++h)
#pragma unroll
            for (int e = 0; e < 4; ++e)
                patch[(8 * h + 4 * c.g + e) * 32 + c.l32] = y[h][e];
        // all four rows read, finished and packed before the first store: a
        // store's data registers cannot be overwritten until the store has
        // read them, so reusing them for the next row's patch read would
        // wait out each store's whole latency
        f32x4 w[4];
        epi_u32x2 cp[4];
#pragma unroll
        for (int t = 0; t < 4; ++t)
            w[t] = *reinterpret_cast<const f32x4 *>(patch + (8 * t + (lane >> 3)) * 32 + 4 * cq);
#pragma unroll
        for (int t = 0; t < 4; ++t) {
            const f32x4 y = epi_apply4(d.ep, w[t], b4, r[t], s4, alpha);
            if (d.ep.ycopy)
                cp[t] = epi_bf16x4(y);
            w[t] = epi_pack4(d.ep, y);
        }
#pragma unroll
        for (int t = 0; t < 4; ++t)
            if (col_ok && mb + 8 * t < M) {
                epi_store_packed4(d.ep, d.Y, (int64_t)(mb + 8 * t) * N + n, w[t], true);
                epi_copy4(d.ep, (int64_t)(mb + 8 * t) * N + n, cp[t], true);
            }
    };

    if (S > 1 && d.cnt) {
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
        constexpr int G4 = MSUB * NSUB * 4;  // 16-byte groups per thread
        float *const tp = d.part + (int64_t)tile * S * (BM * BN);
        float *const mine = tp + (int64_t)part * (BM * BN);
#pragma unroll
        for (int i = 0; i < MSUB; ++i) {
            int ex[16];
            shifts(i, ex);
#pragma unroll
            for (int j = 0; j < NSUB; ++j)
#pragma unroll
                for (int h = 0; h < 4; ++h)
                    st_coherent(mine + (((i * NSUB + j) * 4 + h) * THREADS + tid) * 4,
                                group(i, j, h, ex));
            __builtin_amdgcn_sched_barrier(0);
        }
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        __syncthreads();  // the tile's stores are complete
        // (the flag sits in the scale ring, clear of the store patches)
        int *const flag = reinterpret_cast<int *>(c.sring);
        if (tid == 0)
            *flag = __hip_atomic_fetch_add(d.cnt + tile, 1, __ATOMIC_RELAXED,
                                           __HIP_MEMORY_SCOPE_AGENT);
        __syncthreads();
        if (*flag != S - 1)
            return;
        // Every part, this one included, has stored its partial tile: the
        // sum is read back from memory, one 32 x 32 tile (4 groups of every
        // part, up to 16 loads of 16 bytes) per round trip, and added in part
        // order.
        static_assert(G4 % 4 == 0, "whole 32 x 32 tiles per batch");
#pragma unroll
        for (int gb = 0; gb < G4; gb += 4) {
            f32x4 v[MAXSPLIT][4];
#pragma unroll
            for (int q = 0; q < MAXSPLIT; ++q)
#pragma unroll
                for (int u = 0; u < 4; ++u)
                    if (q < S)
                        v[q][u] = ld_coherent(tp + (int64_t)q * (BM * BN) +
                                              ((gb + u) * THREADS + tid) * 4);
#pragma unroll
            for (int u = 0; u < 4; ++u)
#pragma unroll
                for (int q = 1; q < MAXSPLIT; ++q)
                    if (q < S)
                        v[0][u] += v[q][u];
            const f32x4 y[4] = {v[0][0], v[0][1], v[0][2], v[0][3]};
            store_tile(gb / (NSUB * 4), (gb / 4) % NSUB, y);
            __builtin_amdgcn_sched_barrier(0);
        }
        return;
    }

#pragma unroll
    for (int i = 0; i < MSUB; ++i) {
        int ex[16];
        shifts(i, ex);
#pragma unroll
        for (int j = 0; j < NSUB; ++j) {
            f32x4 y[4];
#pragma unroll
            for (int h = 0; h < 4; ++h)
                y[h] = group(i, j, h, ex);
            store_tile(i, j, y);
        }
        // one row block at a time: hoisting every block's loads would
        // need more registers than the accumulators leave
        __builtin_amdgcn_sched_barrier(0);
    }
}

// Sum of the S plain partial outputs P[s][M][N] of a split layer, in part
// order (the same sum as the in-kernel reduction): Y = ((P0 + P1) + P2) ...
// Loads go out eight parts at a time so that a thread has eight in flight.
struct SumJob {
    const float *P;
    float *Y;
    int S, v4;
    int64_t count;  // outputs per part, in 4-element groups if v4
    int64_t N;
    Epilogue ep;    // applied to the sum
};
struct SumArgs {
    SumJob j[QL_MAX_GROUP];
    int64_t begin[QL_MAX_GROUP + 1];
    int n;
};

template <typename T>
__device__ inline T sum_parts(const T *p, int S, int64_t count)
{
    T y = p[0];
    int q = 1;
    for (; q + 8 <= S; q += 8) {
        T v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u)
            v[u] = p[(q + u) * count];
#pragma unroll
        for (int u = 0; u < 8; ++u)
            y += v[u];
    }
    for (; q < S; ++q)
        y += p[q * count];
    return y;
}

// One launch for the split layers of a call: flat index space over every
// job's outputs, 4-element groups for jobs that allow them (N % 4 == 0, Y
// aligned for one 16-byte fp32 or 8-byte bf16 store, bias, residual and
// steering direction 16-byte aligned), single elements otherwise; each
// layer's epilogue is applied to its sums.
__global__ __launch_bounds__(256) void split_sum_kernel(const SumArgs a)
{
    const int64_t stride = (int64_t)gridDim.x * 256;
    for (int64_t x = (int64_t)blockIdx.x * 256 + threadIdx.x; x < a.begin[a.n]; x += stride) {
        int ji = 0;
#pragma unroll
        for (int i = 1; i < QL_MAX_GROUP; ++i)
            if (i < a.n && x >= a.begin[i])
                ji = i;
        const SumJob &jb = a.j[ji];
        const int64_t i = x - a.begin[ji];
        // the column is needed only by the per-column terms
        const bool col = jb.ep.bias || jb.ep.steer;
        if (jb.v4) {
            const f32x4 y = sum_parts(reinterpret_cast<const f32x4 *>(jb.P) + i, jb.S, jb.count);
            const int n = col ? (int)((4 * i) % jb.N) : 0;
            epi_store4(jb.ep, jb.Y, 4 * i, n, y, true);
        } else {
            const int n = col ? (int)(i % jb.N) : 0;
            epi_store(jb.ep, jb.Y, i, n, sum_parts(jb.P + i, jb.S, jb.count));
        }
    }
}

}  // namespace

hipError_t launch_split_sum(const SplitSum *sums, int n, hipStream_t stream)
{
    SumArgs a{};
    int64_t total = 0;
    for (int i = 0; i < n; ++i) {
        const SplitSum &q = sums[i];
        const bool v4 = q.N % 4 == 0 && ((uintptr_t)q.Y & (q.ep.ybf16 ? 7 : 15)) == 0 &&
                        ((uintptr_t)q.ep.bias & 15) == 0 && ((uintptr_t)q.ep.resid & 15) == 0 &&
                        ((uintptr_t)q.ep.steer & 15) == 0;
        const int64_t count = v4 ? q.M * q.N / 4 : q.M * q.N;
        a.j[i] = SumJob{q.P, q.Y, q.S, v4 ? 1 : 0, count, q.N, q.ep};
        a.begin[i] = total;
        total += count;
    }
    for (int i = n; i <= QL_MAX_GROUP; ++i)
        a.begin[i] = total;
    a.n = n;
    if (total == 0)
        return hipSuccess;
    const unsigned grid = (unsigned)std::min<int64_t>((total + 255) / 256, 4096);
    hipLaunchKernelGGL(split_sum_kernel, dim3(grid), dim3(256), 0, stream, a);
    return hipGetLastError();
}

int wide_tile_bm() { return BM; }
int wide_tile_bn() { return BN; }
int wide_max_split() { return MAXSPLIT; }
int wide_wgs_per_cu(int fmt)
{
    return fmt == QL_FMT_F16 ? wgs_per_cu<QL_FMT_F16>() : WGS_PER_CU;
}

hipError_t launch_qgemm_wide(int fmt, const GroupArgs &args, hipStream_t stream)
{
    dim3 grid((unsigned)args.total_tiles), block(THREADS);
    bool epi = false;
    for (int i = 0; i < args.n; ++i) {
        const Epilogue &e = args.d[i].ep;
        epi = epi || epi_active(e);
    }
    auto go = [&](auto kernel) { hipLaunchKernelGGL(kernel, grid, block, 0, stream, args); };
    if (fmt == QL_FMT_INT8)
        epi ? go(qgemm_wide_kernel<QL_FMT_INT8, true>) : go(qgemm_wide_kernel<QL_FMT_INT8, false>);
    else if (fmt == QL_FMT_Q4)
        epi ? go(qgemm_wide_kernel<QL_FMT_Q4, true>) : go(qgemm_wide_kernel<QL_FMT_Q4, false>);
    else
        epi ? go(qgemm_wide_kernel<QL_FMT_F16, true>) : go(qgemm_wide_kernel<QL_FMT_F16, false>);
    return hipGetLastError();
}

}  // namespace qlk
