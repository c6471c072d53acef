// The steering injection of the paper's Eq. 2 (Methodology, additive
// injection) as an operation of its own: h[m][n] += alpha * hnorm * d[n] on
// the residual stream h [M][N] (fp32, in place), d a unit direction, hnorm
// the layer's mean residual norm, alpha read from device memory at run time
// so that a captured graph picks up a new strength at every replay.  At
// alpha = 0 nothing is written: h stays bit for bit.  (The same term is
// available fused into a linear layer's epilogue.)
//
// Bound: HBM (8 bytes read and 4 written per element when alpha != 0).
// One thread per 4 consecutive elements of a row when N % 4 == 0 and the
// pointers allow 16-byte access, one per element otherwise.
#include <algorithm>

#include "internal.h"

namespace qlk {
namespace {

typedef float f32x4_t __attribute__((ext_vector_type(4)));

__global__ __launch_bounds__(256) void steer_kernel(float *__restrict__ h, int64_t M, int64_t N,
                                                    const float *__restrict__ dir, float hnorm,
                                                    const float *__restrict__ strength, bool vec)
{
    const float alpha = *strength;
    if (alpha == 0.0f)
        return;
    const float c = alpha * hnorm;
    const int64_t stride = (int64_t)gridDim.x * 256;
    if (vec) {
        const int64_t n4 = N / 4, total = M * n4;
        for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < total; i += stride) {
            const int64_t col = (i % n4) * 4;
            f32x4_t v = reinterpret_cast<f32x4_t *>(h)[i];
            const f32x4_t d = *reinterpret_cast<const f32x4_t *>(dir + col);
#pragma unroll
            for (int q = 0; q < 4; ++q)
                v[q] += c * d[q];
            reinterpret_cast<f32x4_t *>(h)[i] = v;
        }
    } else {
        const int64_t total = M * N;
        for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < total; i += stride)
            h[i] += c * dir[i % N];
    }
}

}  // namespace

hipError_t launch_steer(float *h, int64_t M, int64_t N, const float *dir, float hnorm,
                        const float *strength, hipStream_t stream)
{
    const bool vec = N % 4 == 0 && ((uintptr_t)h & 15) == 0 && ((uintptr_t)dir & 15) == 0;
    const int64_t items = vec ? M * (N / 4) : M * N;
    const unsigned grid = (unsigned)std::min<int64_t>((items + 255) / 256, 8192);
    hipLaunchKernelGGL(steer_kernel, dim3(grid), dim3(256), 0, stream, h, M, N, dir, hnorm,
                       strength, vec);
    return hipGetLastError();
}

}  // namespace qlk
