// W8A8 forward: per-token int8 activations against int8 block-quantized
// weights on the int8 matrix cores.
//
// Paper (Methodology, the 8-bit-arithmetic mode of the runtime; Table II):
// activations are quantized alongside the weights and the products run in
// 8-bit integers.  With per-token activation scales s_x[m] and the weights'
// per-block scales s[n][b]:
//
//   Y[m][n] = s_x[m] * sum_b s[n][b] * D_b[m][n],
//   D_b[m][n] = sum_{k in block b} q[m][k] * c[n][k]      (exact, int32)
//
// Each 32 x 32 output tile of a 32-k block is one v_mfma_i32_32x32x32_i8
// (exact), converted and folded into an fp32 accumulator with one FMA per
// output (scale of the lane's column); s_x[m] and the layer epilogue are
// applied at the store.  The per-block rescale is what bounds this kernel:
// 16 outputs per lane per MFMA cost two VALU instructions each, several
// times the MFMA's own issue time.
//
// Tiling: 128 x 128 outputs per workgroup of 4 wavefronts (64 x 64 each,
// 2 x 2 MFMA tiles), K in stages of 64 (two blocks) double-buffered in LDS
// through registers; rows padded to 80 bytes so that the 32 rows an operand
// read touches spread over the LDS banks.
#include "epilogue.h"
#include "internal.h"

namespace qlk {
namespace {

typedef int i32x4 __attribute__((ext_vector_type(4)));
typedef int i32x16 __attribute__((ext_vector_type(16)));

constexpr int BM = 128, BN = 128, BK = 64;
constexpr int THREADS = 256;
constexpr int ROW = 80;                    // LDS bytes per tile row (64 + 16)
constexpr int TILE = BM * ROW;             // one operand tile
constexpr int STAGE = 2 * TILE + 2 * BN * 4;  // X tile, W tile, scales [2][BN] fp32
constexpr int GROUP_M = 8;                 // row tiles that share a column sweep
static_assert(BM == BN, "one chunk mapping serves both operand tiles");

__device__ inline float f16_value(uint16_t bits)
{
    return (float)__builtin_bit_cast(_Float16, bits);
}

// Workgroup p runs on XCD p % 8; give each XCD a contiguous range of the T
// tiles so that neighbouring tiles share an L2.
__device__ inline int xcd_tile(int p, int T)
{
    const int q = T >> 3, r = T & 7;
    const int xcd = p & 7, idx = p >> 3;
    return xcd < r ? xcd * (q + 1) + idx : r * (q + 1) + (xcd - r) * q + idx;
}

__global__ __launch_bounds__(THREADS, 2) void qgemm_w8a8_kernel(const W8Args a)
{
    __shared__ __align__(16) uint8_t lds[2 * STAGE];
    const int T = a.tiles_m * a.tiles_n;
    const int tile = xcd_tile((int)blockIdx.x, T);
    const int per_group = GROUP_M * a.tiles_n;
    const int first_m = (tile / per_group) * GROUP_M;
    const int gsz = min(a.tiles_m - first_m, GROUP_M);
    const int within = tile % per_group;
    const int m0 = (first_m + within % gsz) * BM, n0 = (within / gsz) * BN;

    const int M = a.M, N = a.N, K = a.K, nb = K / 32;
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    const int wm = (wave >> 1) * 64, wn = (wave & 1) * 64;  // the wave's 64 x 64
    const int l32 = lane & 31, hi = lane >> 5;

    // staging: thread t moves 16-byte chunks c = t and t + 256 of each
    // operand tile (row c / 4, bytes 16 (c % 4) of the stage's 64) and the
    // scale of column t % 128, block t / 128 of the stage
    int crow[2], ccol[2];
#pragma unroll
    for (int i = 0; i < 2; ++i) {
        crow[i] = (tid + THREADS * i) >> 2;
        ccol[i] = 16 * ((tid + THREADS * i) & 3);
    }
    const int scol = tid & (BN - 1), sblk = tid >> 7;
    i32x4 px[2], pw[2];
    float ps;
    auto fetch = [&](int s) {
        const int k0 = s * BK;
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            const int k = k0 + ccol[i];
            const int mr = m0 + crow[i], nr = n0 + crow[i];
            px[i] = mr < M && k < K
                        ? *reinterpret_cast<const i32x4 *>(a.qx + (int64_t)mr * K + k)
                        : i32x4{0, 0, 0, 0};
            pw[i] = nr < N && k < K
                        ? *reinterpret_cast<const i32x4 *>(a.codes + (int64_t)nr * K + k)
                        : i32x4{0, 0, 0, 0};
        }
        const int b = 2 * s + sblk, n = n0 + scol;
        ps = n < N && b < nb ? f16_value(a.scales[(int64_t)n * nb + b]) : 0.0f;
    };
    auto put = [&](int buf) {
        uint8_t *st = lds + buf * STAGE;
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            *reinterpret_cast<i32x4 *>(st + crow[i] * ROW + ccol[i]) = px[i];
            *reinterpret_cast<i32x4 *>(st + TILE + crow[i] * ROW + ccol[i]) = pw[i];
        }
        reinterpret_cast<float *>(st + 2 * TILE)[sblk * BN + scol] = ps;
    };

    float acc[2][2][16];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r)
                acc[i][j][r] = 0.0f;

    const int nsteps = (K + BK - 1) / BK;
    fetch(0);
    put(0);
    __syncthreads();
    for (int s = 0; s < nsteps; ++s) {
        if (s + 1 < nsteps)
            fetch(s + 1);
        const uint8_t *st = lds + (s & 1) * STAGE;
        const float *sc = reinterpret_cast<const float *>(st + 2 * TILE);
#pragma unroll
        for (int blk = 0; blk < 2; ++blk) {
            // lane (l32, hi) holds row l32 of the A tile and column l32 of
            // the B tile, k = 16 hi .. 16 hi + 15 of the block
            i32x4 av[2], bv[2];
            float sw[2];
#pragma unroll
            for (int i = 0; i < 2; ++i)
                av[i] = *reinterpret_cast<const i32x4 *>(st + (wm + 32 * i + l32) * ROW +
                                                         32 * blk + 16 * hi);
#pragma unroll
            for (int j = 0; j < 2; ++j) {
                bv[j] = *reinterpret_cast<const i32x4 *>(st + TILE + (wn + 32 * j + l32) * ROW +
                                                         32 * blk + 16 * hi);
                sw[j] = sc[blk * BN + wn + 32 * j + l32];
            }
            i32x16 dv[2][2];
#pragma unroll
            for (int i = 0; i < 2; ++i)
#pragma unroll
                for (int j = 0; j < 2; ++j)
                    dv[i][j] = __builtin_amdgcn_mfma_i32_32x32x32_i8(
                        av[i], bv[j], i32x16{0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0},
                        0, 0, 0);
#pragma unroll
            for (int i = 0; i < 2; ++i)
#pragma unroll
                for (int j = 0; j < 2; ++j)
#pragma unroll
                    for (int r = 0; r < 16; ++r)
                        acc[i][j][r] = __builtin_fmaf(sw[j], (float)dv[i][j][r], acc[i][j][r]);
        }
        if (s + 1 < nsteps)
            put((s + 1) & 1);
        __syncthreads();
    }

    // output (row 8 (r / 4) + 4 hi + r % 4, column l32 of each 32 x 32 tile):
    // times the row's activation scale, then the layer epilogue
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int m = m0 + wm + 32 * i + 8 * (r >> 2) + 4 * hi + (r & 3);
            if (m >= M)
                continue;
            const float sxm = f16_value(a.sx[m]);
#pragma unroll
            for (int j = 0; j < 2; ++j) {
                const int n = n0 + wn + 32 * j + l32;
                if (n < N)
                    epi_store(a.ep, a.Y, (int64_t)m * N + n, n, sxm * acc[i][j][r]);
            }
        }
}

}  // namespace

hipError_t launch_qgemm_w8a8(const W8Args &a, hipStream_t stream)
{
    W8Args b = a;
    b.tiles_m = (a.M + BM - 1) / BM;
    b.tiles_n = (a.N + BN - 1) / BN;
    const int64_t T = (int64_t)b.tiles_m * b.tiles_n;
    if (T <= 0 || T >= ((int64_t)1 << 31))
        return hipErrorInvalidValue;
    hipLaunchKernelGGL(qgemm_w8a8_kernel, dim3((unsigned)T), dim3(THREADS), 0, stream, b);
    return hipGetLastError();
}

}  // namespace qlk
