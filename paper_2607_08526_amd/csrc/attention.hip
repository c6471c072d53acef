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
// tiles of 64, double-buffered in LDS (K row-major, V transposed) through
// registers.
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
constexpr int PAD = 8;             // bf16 elements of padding per LDS row
constexpr int KROW = DH + PAD;     // Ks row: one key
// Vt row: one value channel, 34 words (= 2 mod 32 banks), so that the 16
// rows of one phase of 8-byte operand reads land on distinct banks
constexpr int VROW = BKEY + 4;
constexpr int KBYTES = BKEY * KROW * 2, VBYTES = DH * VROW * 2;
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
    auto kbuf = [&](int i) { return reinterpret_cast<uint16_t *>(lds + i * KBYTES); };
    auto vbuf = [&](int i) { return reinterpret_cast<uint16_t *>(lds + 2 * KBYTES + i * VBYTES); };

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

    // staging: thread t moves rows 2 (t / 8) and 2 (t / 8) + 1 of the K tile,
    // elements 8 (t % 8) .. + 7, and rows 2 (t % 32), 2 (t % 32) + 1 of the V
    // tile, elements 8 (t / 32) .. + 7.  V is written transposed, the two
    // keys of a row pair packed into one 32-bit word; with 32 row pairs per
    // wavefront those writes spread over the LDS banks (8 row pairs per
    // wavefront put every write of an instruction into 8 banks).  Keys at or
    // beyond T repeat key T - 1 (their probabilities are set to 0).
    const int pr = tid >> 3, c8 = 8 * (tid & 7);
    const int vpr = tid & 31, vc8 = 8 * (tid >> 5);
    u32x4 pk[2], pv[2];
    // A tile's rows are read from its first row (a wave-uniform address)
    // plus a per-lane 32-bit byte offset, fixed for full tiles; only the
    // last tile's rows are clamped, lane by lane.
    const uint8_t *const kbase = reinterpret_cast<const uint8_t *>(a.k + seq * a.ldk + h * DH);
    const uint8_t *const vbase = reinterpret_cast<const uint8_t *>(a.v + seq * a.ldv + h * DH);
    const int64_t ktile = (int64_t)BKEY * a.ldk * 2, vtile = (int64_t)BKEY * a.ldv * 2;
    const uint32_t koff = (uint32_t)((2 * pr * a.ldk + c8) * 2), kstep = (uint32_t)(a.ldk * 2);
    const uint32_t voff = (uint32_t)((2 * vpr * a.ldv + vc8) * 2), vstep = (uint32_t)(a.ldv * 2);
    auto fetch_k = [&](int kt) {
        const uint8_t *const t = kbase + kt * ktile;
        uint32_t o[2] = {koff, koff + kstep};
        if ((kt + 1) * BKEY > T)
#pragma unroll
            for (int i = 0; i < 2; ++i)
                o[i] = (uint32_t)(((min(kt * BKEY + 2 * pr + i, T - 1) - kt * BKEY) * a.ldk + c8) * 2);
#pragma unroll
        for (int i = 0; i < 2; ++i)
            pk[i] = *reinterpret_cast<const u32x4 *>(t + o[i]);
    };
    auto fetch_v = [&](int kt) {
        const uint8_t *const t = vbase + kt * vtile;
        uint32_t o[2] = {voff, voff + vstep};
        if ((kt + 1) * BKEY > T)
#pragma unroll
            for (int i = 0; i < 2; ++i)
                o[i] = (uint32_t)(((min(kt * BKEY + 2 * vpr + i, T - 1) - kt * BKEY) * a.ldv + vc8) * 2);
#pragma unroll
        for (int i = 0; i < 2; ++i)
            pv[i] = *reinterpret_cast<const u32x4 *>(t + o[i]);
    };
    auto put_k = [&](uint16_t *ks) {
#pragma unroll
        for (int i = 0; i < 2; ++i)
            *reinterpret_cast<u32x4 *>(ks + (2 * pr + i) * KROW + c8) = pk[i];
    };
    auto put_v = [&](uint16_t *vt) {
        // channel e of the two keys: half e % 2 of word e / 2 of each row,
        // paired by one byte permute (the low half of row 2 vpr first)
#pragma unroll
        for (int e = 0; e < 8; ++e)
            *reinterpret_cast<uint32_t *>(vt + (vc8 + e) * VROW + 2 * vpr) =
                __builtin_amdgcn_perm(pv[1][e >> 1], pv[0][e >> 1],
                                      (e & 1) ? 0x07060302u : 0x05040100u);
    };
    // scores of this lane's query against keys 32 sub + 8 (r / 4) + 4 hf + r % 4
    // (all eight K fragments are read before the first MFMA)
    auto scores = [&](const uint16_t *ks, f32x16 (&sc)[2]) {
        bf16x8 ka[4][2];
#pragma unroll
        for (int s = 0; s < 4; ++s)
#pragma unroll
            for (int sub = 0; sub < 2; ++sub)
                ka[s][sub] = __builtin_bit_cast(
                    bf16x8, *reinterpret_cast<const u32x4 *>(ks + (32 * sub + l32) * KROW +
                                                             16 * s + 8 * hf));
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
    auto tile_pv = [&](auto tailc, int kt, const f32x16 (&sc)[2], const uint16_t *vt) {
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
                const uint16_t *row = vt + (32 * t + l32) * VROW + 16 * kc + 4 * hf;
                const u32x2 lo = *reinterpret_cast<const u32x2 *>(row);
                const u32x2 hi = *reinterpret_cast<const u32x2 *>(row + 8);
                const bf16x8 va = __builtin_bit_cast(bf16x8, u32x4{lo[0], lo[1], hi[0], hi[1]});
                oacc[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                    va, __builtin_bit_cast(bf16x8, pb[kc >> 1][kc & 1]), oacc[t], 0, 0, 0);
            }
    };

    const int nkt = (T + BKEY - 1) / BKEY;
    fetch_k(0);
    fetch_v(0);
    put_k(kbuf(0));
    put_v(vbuf(0));
    if (nkt > 1) {
        fetch_k(1);
        put_k(kbuf(1));
    }
    __syncthreads();
    // one step: tile kt (of parity ODD: its buffers are known at compile
    // time, so LDS addresses fold into offsets), whose scores are in cur (it
    // is full, and tile kt + 1 exists); the scores of tile kt + 1 go to nxt
    auto step = [&](auto oddc, int kt, const f32x16 (&cur)[2], f32x16 (&nxt)[2]) {
        constexpr int P = decltype(oddc)::value ? 1 : 0;
        __syncthreads();  // K of tile kt + 1 and V of tile kt are in LDS
        if (kt + 2 < nkt)
            fetch_k(kt + 2);
        fetch_v(kt + 1);
        tile_max(Flag<false>{}, kt, cur);
        scores(kbuf(P ^ 1), nxt);
        tile_pv(Flag<false>{}, kt, cur, vbuf(P));
        if (kt + 2 < nkt)
            put_k(kbuf(P));
        put_v(vbuf(P ^ 1));
    };
    auto last = [&](auto oddc, int kt, const f32x16 (&cur)[2]) {
        constexpr int P = decltype(oddc)::value ? 1 : 0;
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
