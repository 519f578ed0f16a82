// Float32 rows to a storage type: the optional storage step before a cache
// build or a match, for a caller that holds float32 embeddings.
//
// One wavefront per row, lanes striding over it in 16-byte chunks.  IEEE
// binary16 comes from the hardware conversion (round to nearest-even,
// overflow to +-Inf); bfloat16 and e4m3fn are rounded to nearest-even in
// integer arithmetic from the formats' definitions.  e4m3fn rows get one
// float32 scale each: s = amax / 448 (amax = the largest |x| of the row; s = 1
// when it is not > 0, which includes a row holding NaN), and the codes of
// clamp(x / s, -448, 448).
#include "apc_internal.h"

namespace apc {
namespace {

__device__ inline uint32_t enc_f16(float x)
{
    const _Float16 h = (_Float16)x;
    uint16_t b;
    __builtin_memcpy(&b, &h, 2);
    if (x != x) b = (uint16_t)(((__float_as_uint(x) >> 16) & 0x8000u) | 0x7e00u);   // quiet NaN, sign kept
    return b;
}

__device__ inline uint32_t enc_bf16(float x)
{
    const uint32_t u = __float_as_uint(x);
    if (x != x) return ((u >> 16) | 0x0040u) & 0xffffu;          // quiet NaN, sign and top payload kept
    return (u + 0x7fffu + ((u >> 16) & 1u)) >> 16;                 // nearest-even; a carry may reach +-Inf
}

// e4m3fn code of y (|y| <= 448 or NaN), rounded to nearest-even
__device__ inline uint32_t enc_e4m3(float y)
{
    const uint32_t u = __float_as_uint(y);
    const uint32_t sign = (u >> 24) & 0x80u;
    if (y != y) return sign | 0x7fu;
    const uint32_t a = u & 0x7fffffffu;
    uint32_t code;
    if (a < 0x3c800000u) {
        // below 2^-6: the subnormal codes m 2^-9 (m = 8 is the smallest
        // normal); |y| 512 is exact, rint rounds it to nearest-even
        code = (uint32_t)__builtin_rintf(__uint_as_float(a) * 512.0f);
    } else {
        // keep the top 3 of the 23 mantissa bits, nearest-even (a carry moves
        // into the exponent), and rebias the exponent from 127 to 7
        const uint32_t q = a >> 20, rem = a & 0xfffffu;
        const uint32_t up = rem > 0x80000u || (rem == 0x80000u && (q & 1u)) ? 1u : 0u;
        code = q + up - ((127u - 7u) << 3);
    }
    return sign | code;
}

template <int DT>
__global__ __launch_bounds__(256) void k_quantize_rows(const float* __restrict__ x, int64_t n, int32_t d,
                                                        uint8_t* __restrict__ out, float* __restrict__ scale)
{
    const int lane = threadIdx.x & 63;
    const int64_t r = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (r >= n) return;
    const float* row = x + r * d;
    float s = 1.0f;
    if constexpr (DT == APC_E4M3) {
        float amax = 0.f;
        bool nan = false;
        for (int c = lane * 4; c < d; c += 64 * 4) {
            const float4 v = *reinterpret_cast<const float4*>(row + c);
            const float e[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                nan |= e[i] != e[i];
                amax = __builtin_fmaxf(amax, __builtin_fabsf(e[i]));
            }
        }
#pragma unroll
        for (int m = 32; m >= 1; m >>= 1) amax = __builtin_fmaxf(amax, __shfl_xor(amax, m, 64));
        nan = __any(nan);
        s = nan ? 1.0f : amax / 448.0f;
        if (!(s > 0.f)) s = 1.0f;
        if (lane == 0) scale[r] = s;
    }
    for (int c = lane * 4; c < d; c += 64 * 4) {
        const float4 v = *reinterpret_cast<const float4*>(row + c);
        const float e[4] = {v.x, v.y, v.z, v.w};
        if constexpr (DT == APC_E4M3) {
            uint32_t w = 0;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                float y = e[i] / s;
                if (y == y) y = __builtin_fminf(__builtin_fmaxf(y, -448.0f), 448.0f);
                w |= enc_e4m3(y) << (8 * i);
            }
            *reinterpret_cast<uint32_t*>(out + r * d + c) = w;
        } else {
            uint32_t w[2];
#pragma unroll
            for (int i = 0; i < 2; ++i) {
                const uint32_t lo = DT == APC_F16 ? enc_f16(e[2 * i]) : enc_bf16(e[2 * i]);
                const uint32_t hi = DT == APC_F16 ? enc_f16(e[2 * i + 1]) : enc_bf16(e[2 * i + 1]);
                w[i] = lo | (hi << 16);
            }
            *reinterpret_cast<uint2*>(out + (r * d + c) * 2) = make_uint2(w[0], w[1]);
        }
    }
}

}  // namespace

hipError_t launch_quantize_rows(int dt, int64_t n, int32_t d, const float* x, void* out, float* scale,
                                hipStream_t s)
{
    if (n <= 0) return hipSuccess;
    const dim3 grid((unsigned)((n + 3) / 4)), block(256);
    uint8_t* o = static_cast<uint8_t*>(out);
    switch (dt) {
    case APC_F16: k_quantize_rows<APC_F16><<<grid, block, 0, s>>>(x, n, d, o, scale); break;
    case APC_BF16: k_quantize_rows<APC_BF16><<<grid, block, 0, s>>>(x, n, d, o, scale); break;
    case APC_E4M3: k_quantize_rows<APC_E4M3><<<grid, block, 0, s>>>(x, n, d, o, scale); break;
    default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

}  // namespace apc
