// Fused epilogue of a linear layer, applied by whichever kernel stores a
// final output element (never to split partials): the rest of a DiT block's
// linear -- bias, the feed-forward's GELU, the residual add --
//
//   Y[m][n] = act(P[m][n] + bias[n]) + resid[m][n]          (fp32)
//
// act the identity or the GELU in its exact form x * Phi(x) =
// x * (1 + erf(x / sqrt 2)) / 2, then stored as fp32 or as bf16 (round to
// nearest even, NaN kept quiet).  Elements are addressed by their flat
// index idx = m * N + n and their column n.
#pragma once

#include "internal.h"

namespace qlk {

__device__ inline float epi_gelu(float v)
{
    return 0.5f * v * (1.0f + erff(v * 0.70710678118654752f));
}

__device__ inline float epi_value(const Epilogue &e, int64_t idx, int n, float v)
{
    if (e.bias)
        v += e.bias[n];
    if (e.act == QL_ACT_GELU)
        v = epi_gelu(v);
    if (e.resid)
        v += e.resid[idx];
    return v;
}

__device__ inline uint32_t epi_bf16(float v)
{
    const uint32_t u = __float_as_uint(v);
    if ((u & 0x7FFFFFFFu) > 0x7F800000u)
        return 0x7FC0u;
    return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
}

// one element
__device__ inline void epi_store(const Epilogue &e, float *Y, int64_t idx, int n, float v)
{
    v = epi_value(e, idx, n, v);
    if (e.ybf16)
        reinterpret_cast<uint16_t *>(Y)[idx] = (uint16_t)epi_bf16(v);
    else
        Y[idx] = v;
}

// Whether four consecutive elements of a row (n % 4 == 0, n + 3 < N) can go
// out as one 16-byte (fp32) or 8-byte (bf16) store.
__device__ inline bool epi_vec_ok(const Epilogue &e, const float *Y, int64_t N)
{
    return (N & 3) == 0 && ((uintptr_t)Y & (e.ybf16 ? 7 : 15)) == 0;
}

// elements idx .. idx + 3 (columns n .. n + 3) with one store, streaming
// (nontemporal) when nt
template <typename V4>
__device__ inline void epi_store4(const Epilogue &e, float *Y, int64_t idx, int n, V4 v, bool nt)
{
#pragma unroll
    for (int q = 0; q < 4; ++q)
        v[q] = epi_value(e, idx + q, n + q, v[q]);
    if (e.ybf16) {
        typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
        const u32x2 w = {epi_bf16(v[0]) | (epi_bf16(v[1]) << 16),
                         epi_bf16(v[2]) | (epi_bf16(v[3]) << 16)};
        u32x2 *dst = reinterpret_cast<u32x2 *>(reinterpret_cast<uint16_t *>(Y) + idx);
        if (nt)
            __builtin_nontemporal_store(w, dst);
        else
            *dst = w;
    } else {
        V4 *dst = reinterpret_cast<V4 *>(Y + idx);
        if (nt)
            __builtin_nontemporal_store(v, dst);
        else
            *dst = v;
    }
}

}  // namespace qlk
