// Measurement helpers for the benchmark (not part of the library's product
// path):
//   qlbench_read  a plain streaming read of n16 16-byte chunks, the fastest
//                 way this GPU moves bytes from HBM into the shader cores.
//                 Its time per call, for a buffer of the size of one weight
//                 matrix, is the practical ceiling that a weight-streaming
//                 forward kernel is compared against (it includes the same
//                 per-launch overhead).  Each thread reads one chunk; nothing
//                 is written unless the (impossible) sentinel value appears.
//                 Also the reference of the FETCH_SIZE counter: bytes read,
//                 none written.
//   qlbench_fill  a plain streaming write of n16 16-byte chunks (whole
//                 lines, nothing read): the reference of WRITE_SIZE.
//   qlbench_mark  an empty kernel of `id` workgroups of 64 threads, launched
//                 between the measured calls of a counter run so that the
//                 per-dispatch counter records can be split by grid size.
#include <hip/hip_runtime.h>
#include <stdint.h>

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__global__ __launch_bounds__(256) void read_ceiling_kernel(const u32x4 *__restrict__ p, int64_t n16,
                                                           uint32_t *__restrict__ sink)
{
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= n16)
        return;
    const u32x4 v = __builtin_nontemporal_load(p + i);
    if ((v.x ^ v.y ^ v.z ^ v.w) == 0x9E3779B9u && v.x == 0x7F4A7C15u)
        sink[0] = v.y;
}

extern "C" int qlbench_read(const void *buf, int64_t bytes, void *sink, hipStream_t stream)
{
    if (!buf || !sink || bytes <= 0 || (bytes & 15) || ((uintptr_t)buf & 15))
        return 1;
    const int64_t n16 = bytes / 16;
    const int64_t blocks = (n16 + 255) / 256;
    if (blocks >= ((int64_t)1 << 31))
        return 1;
    hipLaunchKernelGGL(read_ceiling_kernel, dim3((unsigned)blocks), dim3(256), 0, stream,
                       (const u32x4 *)buf, n16, (uint32_t *)sink);
    return hipGetLastError() == hipSuccess ? 0 : 6;
}

__global__ __launch_bounds__(256) void fill_kernel(u32x4 *__restrict__ p, int64_t n16, uint32_t v)
{
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i < n16)
        __builtin_nontemporal_store(u32x4{v, v, v, v}, p + i);
}

extern "C" int qlbench_fill(void *buf, int64_t bytes, uint32_t value, hipStream_t stream)
{
    if (!buf || bytes <= 0 || (bytes & 15) || ((uintptr_t)buf & 15))
        return 1;
    const int64_t n16 = bytes / 16;
    const int64_t blocks = (n16 + 255) / 256;
    if (blocks >= ((int64_t)1 << 31))
        return 1;
    hipLaunchKernelGGL(fill_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, (u32x4 *)buf,
                       n16, value);
    return hipGetLastError() == hipSuccess ? 0 : 6;
}

__global__ __launch_bounds__(64) void mark_kernel(uint32_t *__restrict__ sink, int id)
{
    if (id < 0)
        sink[0] = (uint32_t)id;  // never: keeps the kernel from being empty
}

extern "C" int qlbench_mark(int id, void *sink, hipStream_t stream)
{
    if (id <= 0 || id > 65535 || !sink)
        return 1;
    hipLaunchKernelGGL(mark_kernel, dim3((unsigned)id), dim3(64), 0, stream, (uint32_t *)sink, id);
    return hipGetLastError() == hipSuccess ? 0 : 6;
}
