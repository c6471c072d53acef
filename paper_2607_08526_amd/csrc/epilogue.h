// Fused epilogue of a linear layer, applied by whichever kernel stores a
// final output element (never to split partials): the rest of a DiT block's
// linear -- bias, the feed-forward's GELU, the residual add -- and the
// steering injection of the paper's Eq. 2 on the block's output,
//
//   Y[m][n] = act(P[m][n] + bias[n]) + resid[m][n] + alpha hnorm d[n]  (fp32)
//
// with alpha read from device memory by every launch (a captured graph
// picks up a new strength without re-capture); at alpha = 0 the term is
// skipped, so the output is bit for bit the unsteered one.
//
// act the identity or the GELU in its exact (erf) form x * Phi(x) =
// x * (1 + erf(x / sqrt 2)) / 2, then stored as fp32 or as bf16 (round to
// nearest even, NaN kept quiet); an fp32 output may also be stored as a
// bf16 copy (the next linear layer's input, when Y is a residual stream).
// Elements are addressed by their flat index idx = m * N + n and their
// column n.
#pragma once

#include "internal.h"

namespace qlk {

// GELU x * Phi(x) with Phi(x) = erfc(-x / sqrt 2) / 2 and, for z >= 0,
// erfc(z) = t (a1 + t (a2 + t (a3 + t (a4 + t a5)))) exp(-z^2),
// t = 1 / (1 + p z): the rational approximation of Abramowitz & Stegun
// 7.1.26 (after Hastings), absolute error at most 1.5e-7, so |error| of
// the GELU stays below about 2e-7 |x| with fp32 rounding.  Branch-free, so
// that the fully unrolled store code stays small.
__device__ inline float epi_gelu(float v)
{
    const float z = __builtin_fabsf(v) * 0.70710678118654752f;
    const float t = __builtin_amdgcn_rcpf(__builtin_fmaf(0.3275911f, z, 1.0f));
    float q = __builtin_fmaf(t, 1.061405429f, -1.453152027f);
    q = __builtin_fmaf(t, q, 1.421413741f);
    q = __builtin_fmaf(t, q, -0.284496736f);
    q = __builtin_fmaf(t, q, 0.254829592f);
    q = q * t * __expf(-z * z);  // erfc(|x| / sqrt 2)
    return v * (v >= 0.0f ? 1.0f - 0.5f * q : 0.5f * q);
}

__device__ inline float epi_value(const Epilogue &e, int64_t idx, int n, float v)
{
    if (e.bias)
        v += e.bias[n];
    if (e.act == QL_ACT_GELU)
        v = epi_gelu(v);
    if (e.resid)
        v += e.resid[idx];
    if (e.steer) {
        const float a = *e.strength;
        if (a != 0.0f)
            v += (a * e.hnorm) * e.steer[n];
    }
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
    if (e.ycopy)
        e.ycopy[idx] = (uint16_t)epi_bf16(v);
}

// Whether four consecutive elements of a row (n % 4 == 0, n + 3 < N) can be
// handled as one group: one 16-byte (fp32) or 8-byte (bf16) store, and
// 16-byte loads of the bias and residual.
__host__ __device__ inline bool epi_vec_ok(const Epilogue &e, const float *Y, int64_t N)
{
    return (N & 3) == 0 && ((uintptr_t)Y & (e.ybf16 ? 7 : 15)) == 0 &&
           ((uintptr_t)e.bias & 15) == 0 && ((uintptr_t)e.resid & 15) == 0 &&
           ((uintptr_t)e.steer & 15) == 0 && ((uintptr_t)e.ycopy & 7) == 0;
}

// bf16 bit patterns of four fp32 values, packed in two words
typedef uint32_t epi_u32x2 __attribute__((ext_vector_type(2)));
template <typename V4>
__device__ inline epi_u32x2 epi_bf16x4(V4 v)
{
    return epi_u32x2{epi_bf16(v[0]) | (epi_bf16(v[1]) << 16),
                     epi_bf16(v[2]) | (epi_bf16(v[3]) << 16)};
}

// the bf16 copy of four finished fp32 elements idx .. idx + 3 (a no-op
// without a copy)
__device__ inline void epi_copy4(const Epilogue &e, int64_t idx, epi_u32x2 b, bool nt)
{
    if (e.ycopy) {
        epi_u32x2 *dst = reinterpret_cast<epi_u32x2 *>(e.ycopy + idx);
        if (nt)
            __builtin_nontemporal_store(b, dst);
        else
            *dst = b;
    }
}

// the steering term of four consecutive columns n .. n + 3 (zero, and not
// to be added, when alpha is 0: see epi_apply4)
template <typename V4>
__device__ inline V4 epi_steer4(const Epilogue &e, int n, float &alpha)
{
    V4 s4 = {0.f, 0.f, 0.f, 0.f};
    alpha = 0.0f;
    if (e.steer) {
        alpha = *e.strength;
        if (alpha != 0.0f) {
            const float c = alpha * e.hnorm;
            s4 = *reinterpret_cast<const V4 *>(e.steer + n);
#pragma unroll
            for (int q = 0; q < 4; ++q)
                s4[q] = c * s4[q];
        }
    }
    return s4;
}

// the epilogue of four consecutive elements, their bias, residual and
// steering values already loaded (b4, r4, s4: ignored when the layer has
// none, s4 also when alpha is 0)
template <typename V4>
__device__ inline V4 epi_apply4(const Epilogue &e, V4 v, V4 b4, V4 r4, V4 s4, float alpha)
{
    if (e.bias)
        v += b4;
    if (e.act == QL_ACT_GELU) {
#pragma unroll
        for (int q = 0; q < 4; ++q)
            v[q] = epi_gelu(v[q]);
    }
    if (e.resid)
        v += r4;
    if (alpha != 0.0f)
        v += s4;
    return v;
}

// store of four finished elements idx .. idx + 3, streaming (nontemporal)
// when nt
template <typename V4>
__device__ inline void epi_put4(const Epilogue &e, float *Y, int64_t idx, V4 v, bool nt)
{
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

// the store of epi_put4 split in two: the value as stored (fp32, or bf16
// packed in the low 8 bytes), then the store itself
template <typename V4>
__device__ inline V4 epi_pack4(const Epilogue &e, V4 v)
{
    if (e.ybf16) {
        V4 w = v;
        w[0] = __uint_as_float(epi_bf16(v[0]) | (epi_bf16(v[1]) << 16));
        w[1] = __uint_as_float(epi_bf16(v[2]) | (epi_bf16(v[3]) << 16));
        return w;
    }
    return v;
}

template <typename V4>
__device__ inline void epi_store_packed4(const Epilogue &e, float *Y, int64_t idx, V4 w, bool nt)
{
    if (e.ybf16) {
        typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
        const u32x2 b = {__float_as_uint(w[0]), __float_as_uint(w[1])};
        u32x2 *dst = reinterpret_cast<u32x2 *>(reinterpret_cast<uint16_t *>(Y) + idx);
        if (nt)
            __builtin_nontemporal_store(b, dst);
        else
            *dst = b;
    } else {
        V4 *dst = reinterpret_cast<V4 *>(Y + idx);
        if (nt)
            __builtin_nontemporal_store(w, dst);
        else
            *dst = w;
    }
}

// elements idx .. idx + 3 (columns n .. n + 3) of a group that epi_vec_ok
// allows, loads included
template <typename V4>
__device__ inline void epi_store4(const Epilogue &e, float *Y, int64_t idx, int n, V4 v, bool nt)
{
    V4 b4 = {0.f, 0.f, 0.f, 0.f}, r4 = b4;
    if (e.bias)
        b4 = *reinterpret_cast<const V4 *>(e.bias + n);
    if (e.resid)
        r4 = *reinterpret_cast<const V4 *>(e.resid + idx);
    float alpha;
    const V4 s4 = epi_steer4<V4>(e, n, alpha);
    const V4 y = epi_apply4(e, v, b4, r4, s4, alpha);
    epi_put4(e, Y, idx, y, nt);
    if (e.ycopy)
        epi_copy4(e, idx, epi_bf16x4(y), nt);
}

}  // namespace qlk
