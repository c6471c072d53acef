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
constexpr int STAGE = (BKEY * KROW + DH * VROW) * 2;  // bytes

typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

// two fp32 values rounded to nearest even bf16, packed (v_cvt_pk_bf16_f32)
__device__ inline uint32_t pack_bf16(float lo, float hi)
{
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{lo, hi}, bf16x2));
}

__global__ __launch_bounds__(THREADS, 2) void attention_kernel(const AttnArgs a)
{
    __shared__ __align__(16) uint8_t lds[2 * STAGE];
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    const int l32 = lane & 31, hf = lane >> 5;
    const int bh = blockIdx.y, b = bh / a.H, h = bh - b * a.H;
    const int T = a.T;
    const int64_t seq = (int64_t)b * T;  // first row of this sequence
    const int q = blockIdx.x * BQ + wave * 32 + l32;  // this lane's query

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
    // wavefront put every write of an instruction into 8 banks)
    const int pr = tid >> 3, c8 = 8 * (tid & 7);
    const int vpr = tid & 31, vc8 = 8 * (tid >> 5);
    u32x4 pk[2], pv[2];
    auto fetch = [&](int kt) {
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            const int key = kt * BKEY + 2 * pr + i;
            u32x4 zk = {0u, 0u, 0u, 0u}, zv = zk;
            if (key < T) {
                zk = *reinterpret_cast<const u32x4 *>(a.k + (seq + key) * a.ldk + h * DH + c8);
            }
            const int vkey = kt * BKEY + 2 * vpr + i;
            if (vkey < T)
                zv = *reinterpret_cast<const u32x4 *>(a.v + (seq + vkey) * a.ldv + h * DH + vc8);
            pk[i] = zk;
            pv[i] = zv;
        }
    };
    auto put = [&](int buf) {
        uint16_t *ks = reinterpret_cast<uint16_t *>(lds + buf * STAGE);
        uint16_t *vt = ks + BKEY * KROW;
#pragma unroll
        for (int i = 0; i < 2; ++i)
            *reinterpret_cast<u32x4 *>(ks + (2 * pr + i) * KROW + c8) = pk[i];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const uint32_t lo = (pv[0][e >> 1] >> (16 * (e & 1))) & 0xFFFFu;
            const uint32_t hi = (pv[1][e >> 1] >> (16 * (e & 1))) & 0xFFFFu;
            *reinterpret_cast<uint32_t *>(vt + (vc8 + e) * VROW + 2 * vpr) = lo | (hi << 16);
        }
    };

    f32x16 oacc[2];
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r)
            oacc[t][r] = 0.0f;
    float mrun = -INFINITY, lrun = 0.0f;

    const int nkt = (T + BKEY - 1) / BKEY;
    fetch(0);
    put(0);
    __syncthreads();
    for (int kt = 0; kt < nkt; ++kt) {
        if (kt + 1 < nkt)
            fetch(kt + 1);
        const uint16_t *ks = reinterpret_cast<const uint16_t *>(lds + (kt & 1) * STAGE);
        const uint16_t *vt = ks + BKEY * KROW;

        // scores of this lane's query against keys 32 sub + 8 (r / 4) + 4 hf + r % 4
        f32x16 sc[2];
#pragma unroll
        for (int sub = 0; sub < 2; ++sub) {
            f32x16 acc;
#pragma unroll
            for (int r = 0; r < 16; ++r)
                acc[r] = 0.0f;
#pragma unroll
            for (int s = 0; s < 4; ++s) {
                const bf16x8 ka = __builtin_bit_cast(
                    bf16x8, *reinterpret_cast<const u32x4 *>(ks + (32 * sub + l32) * KROW +
                                                             16 * s + 8 * hf));
                acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka, qb[s], acc, 0, 0, 0);
            }
            sc[sub] = acc;
        }
        // running maximum of the raw scores (keys beyond T excluded; the
        // scale c = scale * log2 e >= 0 is applied inside the exponent:
        // p = 2^(s c - m c))
        const bool tail = (kt + 1) * BKEY > T;
        auto valid = [&](int sub, int r) {
            return kt * BKEY + 32 * sub + 8 * (r >> 2) + 4 * hf + (r & 3) < T;
        };
        float mt = -INFINITY;
#pragma unroll
        for (int sub = 0; sub < 2; ++sub)
#pragma unroll
            for (int r = 0; r < 16; ++r)
                mt = fmaxf(mt, !tail || valid(sub, r) ? sc[sub][r] : -INFINITY);
        mt = fmaxf(mt, __shfl_xor(mt, 32));
        const float c = a.scale_log2e;
        const float mnew = fmaxf(mrun, mt);
        const float alpha = mrun == -INFINITY ? 0.0f : __builtin_amdgcn_exp2f((mrun - mnew) * c);
        mrun = mnew;
        const float mc = mnew * c;
        float ls = 0.0f;
        u32x4 pb[2][2];  // P^T operands: [sub][chunk c], 8 bf16 each
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
                    if (tail) {
                        p0 = valid(sub, r0) ? p0 : 0.0f;
                        p1 = valid(sub, r0 + 1) ? p1 : 0.0f;
                    }
                    ls += p0 + p1;
                    w[e] = pack_bf16(p0, p1);
                }
                pb[sub][ch] = u32x4{w[0], w[1], w[2], w[3]};
            }
        lrun = lrun * alpha + ls;
#pragma unroll
        for (int t = 0; t < 2; ++t)
#pragma unroll
            for (int r = 0; r < 16; ++r)
                oacc[t][r] *= alpha;
        // O^T += V^T P^T over the four 16-key chunks
#pragma unroll
        for (int t = 0; t < 2; ++t)
#pragma unroll
            for (int kc = 0; kc < 4; ++kc) {
                const uint16_t *row = vt + (32 * t + l32) * VROW + 16 * kc + 4 * hf;
                const u32x2 lo = *reinterpret_cast<const u32x2 *>(row);
                const u32x2 hi = *reinterpret_cast<const u32x2 *>(row + 8);
                const bf16x8 va = __builtin_bit_cast(bf16x8, u32x4{lo[0], lo[1], hi[0], hi[1]});
                oacc[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                    va, __builtin_bit_cast(bf16x8, pb[kc >> 1][kc & 1]), oacc[t], 0, 0, 0);
            }
        if (kt + 1 < nkt)
            put((kt + 1) & 1);
        __syncthreads();
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
    const dim3 grid((unsigned)((a.T + BQ - 1) / BQ), (unsigned)(a.B * a.H));
    hipLaunchKernelGGL(attention_kernel, grid, dim3(THREADS), 0, stream, a);
    return hipGetLastError();
}

}  // namespace qlk
