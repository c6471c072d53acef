// Fused self-attention of the DiT block (the GPU path's attention in the
// paper's Methodology; a FlashAttention-class kernel is the open lever it
// names): for every sequence b, head h and query t,
//
//   O[b,t,h,:] = sum_j p_j V[b,j,h,:] / sum_j p_j,
//   p_j = exp(s_j - max_i s_i),  s_j = scale * <Q[b,t,h,:], K[b,j,h,:]>,
//
// over all T keys of the sequence, in one pass with a running maximum and
// sum (the scores never reach memory).  Q, K, V are bf16 rows read with
// strides, so the kernel takes the fused QKV output of the preceding linear
// as it is; O is fp32 or bf16 (the next linear's activations).
//
// Layout on the matrix cores (v_mfma_f32_32x32x16_bf16, head dim 64):
//  * the scores are formed transposed, S^T = K Q^T (A = 32 key rows from
//    LDS, B = the wavefront's 32 queries held in registers), so that lane l
//    holds 16 scores of query l % 32 and lane l ^ 32 the other 16 of the
//    32-key tile: the row maximum and sum need one exchange between the
//    two halves of the wavefront;
//  * the output is accumulated transposed too, O^T += V^T P^T: the B
//    operand is P^T straight from the score registers (rounded to bf16),
//    which hold keys {16c + 4h + i, 16c + 8 + 4h + i : i < 4} of chunk c in
//    lane half h rather than 16c + 8h + i; A = V^T is read from LDS in that
//    same key order, and since both operands use it the contraction over
//    keys is unchanged.  The accumulator of query l % 32 stays in the lanes
//    that hold its softmax state, so the per-query rescaling is local.
// Per workgroup: 128 queries (4 wavefronts x 32) of one (b, h); keys in
// tiles of 64, double-buffered in LDS.  K and V tiles move from global memory
// to LDS with the direct-to-LDS loads (no registers, no LDS write
// instructions), both row-major (one key per 128-byte row, 16-byte chunks
// XOR-swizzled per row against bank conflicts).  The V^T operand is read
// with gfx950's transposing LDS read (ds_read_b64_tr_b16): within each group
// of 16 lanes, result lane 4q + p receives element p of the 8 bytes that
// source lanes q, 4 + q, 8 + q and 12 + q address, so 16 lanes that
// address 4 keys x 4 runs of 4 channels receive 4 keys of one channel each.
#include "internal.h"

namespace qlk {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int DH = 64;             // head dimension
constexpr int BQ = 128, BKEY = 64;  // queries per workgroup, keys per tile
constexpr int THREADS = 256;
constexpr int KBYTES = BKEY * DH * 2, VBYTES = BKEY * DH * 2;  // one tile, row-major
constexpr int TLOADS = KBYTES / 16 / THREADS;  // 16-byte loads per thread per tile
// physical 16-byte chunk = logical ^ swizzle(key row): the K fragment reads
// (32 rows, one chunk) and the transposing V reads (8 rows, two chunk pairs)
// spread over the banks
__device__ inline int kswz(int r) { return (r & 7) ^ ((r >> 3) & 1); }
__device__ inline int vswz(int r) { return ((r >> 1) & 1) << 2; }
// The running maximum m may trail the true one: it moves only when a tile's
// scores exceed it by more than 2^LAZY in the exponent (so p <= 2^LAZY), and
// then the accumulators are rescaled; the quotient O / l is the same for any
// m, and fp32 holds 2^LAZY * T easily.
constexpr float LAZY = 8.0f;

typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

// two fp32 values rounded to nearest even bf16, packed (v_cvt_pk_bf16_f32)
__device__ inline uint32_t pack_bf16(float lo, float hi)
{
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{lo, hi}, bf16x2));
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

typedef short s16x4 __attribute__((ext_vector_type(4)));

// 8 bytes of LDS at byte offset `off` of `base`, transposed across each
// group of 16 lanes (see the header)
__device__ inline u32x2 read_tr(const uint8_t *base, uint32_t off)
{
    const s16x4 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        (__attribute__((address_space(3))) s16x4 *)(base + off));
    return __builtin_bit_cast(u32x2, v);
}

template <bool B>
struct Flag {
    static constexpr bool value = B;
};

// Software pipeline over key tiles: while the softmax of tile j runs on the
// VALU, the matrix cores form the scores of tile j + 1 (their K rows are
// already in LDS), then take tile j's value product.  K and V tiles have
// two LDS buffers each, filled one tile apart: during step j the K buffer
// of tile j (read in step j - 1) receives tile j + 2 and the V buffer of
// tile j - 1 receives tile j + 1, so one barrier per step suffices.
__global__ __launch_bounds__(THREADS, 2) __attribute__((amdgpu_waves_per_eu(2, 2)))
void attention_kernel(const AttnArgs a)
{
    __shared__ __align__(16) uint8_t lds[2 * KBYTES + 2 * VBYTES];
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    const int l32 = lane & 31, hf = lane >> 5;
    // workgroup p runs on XCD p % 8; each XCD takes a contiguous range of
    // (sequence, head) pairs with all their query blocks, so each pair's
    // K and V tiles are fetched into one XCD's L2 and re-read there by its
    // query blocks (round-robin pairs would make every XCD fetch them all)
    const int T = a.T, nq = (T + BQ - 1) / BQ;
    const int G = (int)gridDim.x, p = (int)blockIdx.x;
    const int gq = G >> 3, gr = G & 7, xcd = p & 7, idx = p >> 3;
    const int L = xcd < gr ? xcd * (gq + 1) + idx : gr * (gq + 1) + (xcd - gr) * gq + idx;
    const int bh = L / nq, qblk = L - bh * nq, b = bh / a.H, h = bh - b * a.H;
    const int64_t seq = (int64_t)b * T;  // first row of this sequence
    const int q = qblk * BQ + wave * 32 + l32;  // this lane's query
    auto kbuf = [&](int i) { return lds + i * KBYTES; };
    auto vbuf = [&](int i) { return lds + 2 * KBYTES + i * VBYTES; };

    // the query's B operands: head-dim chunk s, elements 16 s + 8 hf .. + 7
    bf16x8 qb[4];
#pragma unroll
    for (int s = 0; s < 4; ++s) {
        u32x4 v = {0u, 0u, 0u, 0u};
        if (q < T)
            v = *reinterpret_cast<const u32x4 *>(a.q + (seq + q) * a.ldq + h * DH + 16 * s +
                                                 8 * hf);
        qb[s] = __builtin_bit_cast(bf16x8, v);
    }

    // staging: the tile's 512 chunks of 16 bytes (K and V alike), slot
    // i = j * 256 + t for thread t's load j: key row i / 8, physical chunk
    // i % 8, holding logical chunk (i % 8) ^ swizzle(row) of the row.  Offsets
    // are from the tile's first key row (a wave-uniform base); keys at or
    // beyond T repeat key T - 1 in the last tile (their probabilities are set
    // to 0).
    const uint8_t *const kbase = reinterpret_cast<const uint8_t *>(a.k + seq * a.ldk + h * DH);
    const uint8_t *const vbase = reinterpret_cast<const uint8_t *>(a.v + seq * a.ldv + h * DH);
    const int64_t ktile = (int64_t)BKEY * a.ldk * 2, vtile = (int64_t)BKEY * a.ldv * 2;
    auto offs = [&](int kt, int64_t ld, bool isk, uint32_t (&o)[TLOADS]) {
#pragma unroll
        for (int j = 0; j < TLOADS; ++j) {
            const int i = j * THREADS + tid, r = i >> 3;
            const int lc = (i & 7) ^ (isk ? kswz(r) : vswz(r));
            const int key = min(kt * BKEY + r, T - 1) - kt * BKEY;
            o[j] = (uint32_t)((key * ld + 8 * lc) * 2);
        }
    };
    uint32_t kof[TLOADS], vof[TLOADS];  // offsets of a full tile
    offs(0, a.ldk, true, kof);
    offs(0, a.ldv, false, vof);
    auto fetch = [&](int kt, const uint8_t *tbase, int64_t tstep, int64_t ld, bool isk,
                     const uint32_t (&full)[TLOADS], uint8_t *buf) {
        uint32_t o[TLOADS];
#pragma unroll
        for (int j = 0; j < TLOADS; ++j)
            o[j] = full[j];
        if ((kt + 1) * BKEY > T)
            offs(kt, ld, isk, o);
        const uint8_t *const t = tbase + kt * tstep;
#pragma unroll
        for (int j = 0; j < TLOADS; ++j)
            dma16(t, o[j], lds_addr(buf) + (j * THREADS + wave * 64) * 16);
    };
    auto fetch_k = [&](int kt, uint8_t *buf) { fetch(kt, kbase, ktile, a.ldk, true, kof, buf); };
    auto fetch_v = [&](int kt, uint8_t *buf) { fetch(kt, vbase, vtile, a.ldv, false, vof, buf); };
    // the transposed V operand: this lane addresses key 16 kc + 8 u + 4 hf +
    // (lane % 16) / 4 and channels 32 t + 16 ((lane / 16) % 2) + 4 (lane % 4)
    // .. + 3, i.e. unit (8 bytes) 8 t + 4 ((lane / 16) % 2) + lane % 4 of its
    // row; the transpose hands lane l the 4 keys of channel 32 t + l % 32
    const int vkey0 = 4 * hf + ((lane & 15) >> 2);
    const int vunit0 = 4 * ((lane >> 4) & 1) + (lane & 3);
    auto voff = [&](int kc, int u, int t) {
        const int key = 16 * kc + 8 * u + vkey0, unit = 8 * t + vunit0;
        return (uint32_t)(key * 128 + (((unit >> 1) ^ vswz(key)) * 16) + (unit & 1) * 8);
    };
    // scores of this lane's query against keys 32 sub + 8 (r / 4) + 4 hf + r % 4
    // (all eight K fragments are read before the first MFMA)
    auto scores = [&](const uint8_t *ks, f32x16 (&sc)[2]) {
        bf16x8 ka[4][2];
#pragma unroll
        for (int s = 0; s < 4; ++s)
#pragma unroll
            for (int sub = 0; sub < 2; ++sub) {
                const int r = 32 * sub + l32;
                ka[s][sub] = __builtin_bit_cast(
                    bf16x8, *reinterpret_cast<const u32x4 *>(ks + r * 128 +
                                                             ((2 * s + hf) ^ kswz(r)) * 16));
            }
        const f32x16 zero = {};
#pragma unroll
        for (int sub = 0; sub < 2; ++sub)
            sc[sub] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka[0][sub], qb[0], zero, 0, 0, 0);
#pragma unroll
        for (int s = 1; s < 4; ++s)
#pragma unroll
            for (int sub = 0; sub < 2; ++sub)
                sc[sub] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka[s][sub], qb[s], sc[sub], 0,
                                                                  0, 0);
    };

    f32x16 oacc[2];
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r)
            oacc[t][r] = 0.0f;
    float mrun = -INFINITY, lrun = 0.0f;
    const float c = a.scale_log2e;  // p = 2^(s c - m c), c >= 0

    // Softmax of one tile's scores and its value product, in two parts so
    // that the next tile's score MFMAs can be placed between them.  TAIL:
    // the last, partial tile (keys at or beyond T get p = 0).
    float alpha = 0.0f;
    auto tile_max = [&](auto tailc, int kt, const f32x16 (&sc)[2]) {
        constexpr bool TAIL = decltype(tailc)::value;
        auto valid = [&](int sub, int r) {
            return !TAIL || kt * BKEY + 32 * sub + 8 * (r >> 2) + 4 * hf + (r & 3) < T;
        };
        // tile maximum: four independent chains (the compiler forms v_max3)
        float mx[4] = {-INFINITY, -INFINITY, -INFINITY, -INFINITY};
#pragma unroll
        for (int sub = 0; sub < 2; ++sub)
#pragma unroll
            for (int r = 0; r < 16; ++r)
                mx[r & 3] = fmaxf(mx[r & 3], valid(sub, r) ? sc[sub][r] : -INFINITY);
        float mt = fmaxf(fmaxf(mx[0], mx[1]), fmaxf(mx[2], mx[3]));
        mt = fmaxf(mt, __shfl_xor(mt, 32));
        // move the maximum only when some lane of the wavefront needs it
        const bool up = mrun == -INFINITY || (mt - mrun) * c > LAZY;
        const bool any_up = __ballot(up) != 0;
        const float mnew = any_up ? fmaxf(mrun, mt) : mrun;
        alpha = mrun == -INFINITY ? 0.0f : __builtin_amdgcn_exp2f((mrun - mnew) * c);
        mrun = mnew;
        lrun *= alpha;
        if (any_up) {
#pragma unroll
            for (int t = 0; t < 2; ++t)
#pragma unroll
                for (int r = 0; r < 16; ++r)
                    oacc[t][r] *= alpha;
        }
    };
    auto tile_pv = [&](auto tailc, int kt, const f32x16 (&sc)[2], const uint8_t *vt) {
        constexpr bool TAIL = decltype(tailc)::value;
        auto valid = [&](int sub, int r) {
            return !TAIL || kt * BKEY + 32 * sub + 8 * (r >> 2) + 4 * hf + (r & 3) < T;
        };
        const float mc = mrun * c;
        float ls[4];
        u32x4 pb[2][2];  // P^T operands: [sub][chunk], 8 bf16 each
#pragma unroll
        for (int sub = 0; sub < 2; ++sub)
#pragma unroll
            for (int ch = 0; ch < 2; ++ch) {
                uint32_t w[4];
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const int r0 = 8 * ch + 2 * e;
                    float p0 = __builtin_amdgcn_exp2f(__builtin_fmaf(sc[sub][r0], c, -mc));
                    float p1 = __builtin_amdgcn_exp2f(__builtin_fmaf(sc[sub][r0 + 1], c, -mc));
                    if (TAIL) {
                        p0 = valid(sub, r0) ? p0 : 0.0f;
                        p1 = valid(sub, r0 + 1) ? p1 : 0.0f;
                    }
                    ls[e] = sub == 0 && ch == 0 ? p0 + p1 : ls[e] + (p0 + p1);
                    w[e] = pack_bf16(p0, p1);
                }
                pb[sub][ch] = u32x4{w[0], w[1], w[2], w[3]};
            }
        lrun += (ls[0] + ls[1]) + (ls[2] + ls[3]);
        // O^T += V^T P^T over the four 16-key chunks
#pragma unroll
        for (int kc = 0; kc < 4; ++kc)
#pragma unroll
            for (int t = 0; t < 2; ++t) {
                const u32x2 lo = read_tr(vt, voff(kc, 0, t));
                const u32x2 hi = read_tr(vt, voff(kc, 1, t));
                const bf16x8 va = __builtin_bit_cast(bf16x8, u32x4{lo[0], lo[1], hi[0], hi[1]});
                oacc[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                    va, __builtin_bit_cast(bf16x8, pb[kc >> 1][kc & 1]), oacc[t], 0, 0, 0);
            }
    };

    const int nkt = (T + BKEY - 1) / BKEY;
    fetch_k(0, kbuf(0));
    fetch_v(0, vbuf(0));
    if (nkt > 1)
        fetch_k(1, kbuf(1));
    // one step: tile kt (of parity ODD: its buffers are known at compile
    // time, so LDS addresses fold into offsets), whose scores are in cur (it
    // is full, and tile kt + 1 exists); the scores of tile kt + 1 go to nxt.
    // At its start every load issued so far has landed (K of tile kt + 1, V
    // of tile kt: the last issued, one step ago) and every wavefront has
    // finished the previous step, so K's buffer of tile kt (read in step
    // kt - 1) takes tile kt + 2 and V's buffer of tile kt - 1 takes tile
    // kt + 1 while this step reads the other two.
    auto step = [&](auto oddc, int kt, const f32x16 (&cur)[2], f32x16 (&nxt)[2]) {
        constexpr int P = decltype(oddc)::value ? 1 : 0;
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        __syncthreads();
        if (kt + 2 < nkt)
            fetch_k(kt + 2, kbuf(P));
        fetch_v(kt + 1, vbuf(P ^ 1));
        tile_max(Flag<false>{}, kt, cur);
        scores(kbuf(P ^ 1), nxt);
        tile_pv(Flag<false>{}, kt, cur, vbuf(P));
    };
    auto last = [&](auto oddc, int kt, const f32x16 (&cur)[2]) {
        constexpr int P = decltype(oddc)::value ? 1 : 0;
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        __syncthreads();  // V of the last tile is in LDS
        if (nkt * BKEY > T) {
            tile_max(Flag<true>{}, kt, cur);
            tile_pv(Flag<true>{}, kt, cur, vbuf(P));
        } else {
            tile_max(Flag<false>{}, kt, cur);
            tile_pv(Flag<false>{}, kt, cur, vbuf(P));
        }
    };
    // two score buffers in turn (no copies between steps)
    f32x16 sa[2], sb[2];
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();  // K of tiles 0 and 1, V of tile 0 are in LDS
    scores(kbuf(0), sa);
    int kt = 0;
    for (; kt + 2 < nkt; kt += 2) {
        step(Flag<false>{}, kt, sa, sb);
        step(Flag<true>{}, kt + 1, sb, sa);
    }
    if (kt + 1 < nkt) {
        step(Flag<false>{}, kt, sa, sb);
        last(Flag<true>{}, kt + 1, sb);
    } else {
        last(Flag<false>{}, kt, sa);
    }

    // normalize and store: channel 32 t + 8 (r / 4) + 4 hf + r % 4 of query q
    const float inv = 1.0f / (lrun + __shfl_xor(lrun, 32));
    if (q >= T)
        return;
    const int64_t orow = (seq + q) * a.ldo + h * DH;
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
            const int ch = 32 * t + 8 * g + 4 * hf;
            const f32x4_t v = {oacc[t][4 * g] * inv, oacc[t][4 * g + 1] * inv,
                               oacc[t][4 * g + 2] * inv, oacc[t][4 * g + 3] * inv};
            if (a.obf16) {
                uint16_t *o = static_cast<uint16_t *>(a.o) + orow + ch;
                *reinterpret_cast<u32x2 *>(o) = u32x2{pack_bf16(v[0], v[1]), pack_bf16(v[2], v[3])};
            } else {
                *reinterpret_cast<f32x4_t *>(static_cast<float *>(a.o) + orow + ch) = v;
            }
        }
}

}  // namespace

hipError_t launch_attention(const AttnArgs &a, hipStream_t stream)
{
    const dim3 grid((unsigned)((int64_t)(a.T + BQ - 1) / BQ * a.B * a.H));
    hipLaunchKernelGGL(attention_kernel, grid, dim3(THREADS), 0, stream, a);
    return hipGetLastError();
}

}  // namespace qlk
