// Row factors f = 1/|x| for cache entries (build) and queries (each batch).
//
// One wavefront per row: lanes stride over the row in 16-byte chunks
// (coalesced), decode to float32, sum squares, then reduce across the wave
// in a fixed order so the result is deterministic.  For e4m3fn rows the norm
// is that of the codes: the positive row scale cancels in the cosine.
#include "apc_internal.h"

namespace apc {
namespace {

__device__ inline float dec_e4m3(uint32_t c)
{
    uint32_t e = (c >> 3) & 15u, m = c & 7u;
    float v;
    if (e == 15u && m == 7u) return __int_as_float(0x7fc00000);
    if (e == 0u)
        v = (float)m * 0.001953125f;                     // m/8 * 2^-6 = m * 2^-9
    else
        v = __uint_as_float(((e + 120u) << 23) | (m << 20));   // (1 + m/8) * 2^(e - 7)
    return (c & 0x80u) ? -v : v;
}

__device__ inline float dec_bf16(uint32_t h) { return __uint_as_float(h << 16); }

__device__ inline float dec_f16(uint32_t h)
{
    _Float16 x;
    uint16_t b = (uint16_t)h;
    __builtin_memcpy(&x, &b, 2);
    return (float)x;
}

template <int DT>
__device__ inline void accum_chunk(const uint4 v, float& ss, bool& bad)
{
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        if constexpr (DT == APC_F32) {
            float x = __uint_as_float(w[j]);
            bad |= !__builtin_isfinite(x);
            ss = fmaf(x, x, ss);
        } else if constexpr (DT == APC_F16 || DT == APC_BF16) {
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                uint32_t c = (w[j] >> (16 * h)) & 0xffffu;
                float x = DT == APC_F16 ? dec_f16(c) : dec_bf16(c);
                bad |= !__builtin_isfinite(x);
                ss = fmaf(x, x, ss);
            }
        } else {
#pragma unroll
            for (int h = 0; h < 4; ++h) {
                float x = dec_e4m3((w[j] >> (8 * h)) & 0xffu);
                bad |= !__builtin_isfinite(x);
                ss = fmaf(x, x, ss);
            }
        }
    }
}

template <int DT>
__global__ __launch_bounds__(256) void k_row_factors(const uint8_t* __restrict__ rows, int64_t n,
                                                      int64_t row_bytes, const float* __restrict__ scale,
                                                      const int32_t* __restrict__ slot_of_entry,
                                                      int64_t n_slots, float* __restrict__ f,
                                                      BuildStatus* __restrict__ st, uint8_t* __restrict__ rowflags)
{
    const int lane = threadIdx.x & 63;
    const int64_t r = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (r >= n) return;
    const uint8_t* row = rows + r * row_bytes;
    float ss = 0.f;
    bool bad = false;
    for (int64_t off = (int64_t)lane * 16; off < row_bytes; off += 64 * 16)
        accum_chunk<DT>(*reinterpret_cast<const uint4*>(row + off), ss, bad);
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) ss += __shfl_xor(ss, m, 64);
    bad = __any(bad);
    if (lane != 0) return;
    uint32_t flags = 0;
    if (bad || !__builtin_isfinite(ss)) flags |= ST_NONFINITE;
    else if (!(ss > 0.f)) flags |= ST_ZERO;
    if (scale) {
        float s = scale[r];
        if (!(__builtin_isfinite(s) && s > 0.f)) flags |= ST_SCALE;
    }
    if (f) f[r] = flags ? __int_as_float(0x7fc00000) : 1.0f / __builtin_sqrtf(ss);
    if (slot_of_entry) {
        int32_t v = slot_of_entry[r];
        if (v < -1 || (int64_t)v >= n_slots) flags |= ST_SLOT;
    }
    if (rowflags) rowflags[r] = (uint8_t)flags;
    if (st && flags) {
        atomicOr(&st->flags, flags);
        atomicMin(&st->first_bad, (unsigned long long)r);
        atomicAdd(&st->n_bad, 1ull);
    }
}

}  // namespace

hipError_t launch_row_factors(int dt, int64_t n, int32_t d, const void* rows, const float* scale,
                              const int32_t* slot_of_entry, int64_t n_slots, float* f,
                              BuildStatus* st, hipStream_t s, uint8_t* rowflags)
{
    if (n <= 0) return hipSuccess;
    const int64_t row_bytes = (int64_t)d * elem_bytes(dt);
    const dim3 grid((unsigned)((n + 3) / 4)), block(256);
    const uint8_t* r = static_cast<const uint8_t*>(rows);
    switch (dt) {
    case APC_F32: k_row_factors<APC_F32><<<grid, block, 0, s>>>(r, n, row_bytes, scale, slot_of_entry, n_slots, f, st, rowflags); break;
    case APC_F16: k_row_factors<APC_F16><<<grid, block, 0, s>>>(r, n, row_bytes, scale, slot_of_entry, n_slots, f, st, rowflags); break;
    case APC_BF16: k_row_factors<APC_BF16><<<grid, block, 0, s>>>(r, n, row_bytes, scale, slot_of_entry, n_slots, f, st, rowflags); break;
    default: k_row_factors<APC_E4M3><<<grid, block, 0, s>>>(r, n, row_bytes, scale, slot_of_entry, n_slots, f, st, rowflags); break;
    }
    return hipGetLastError();
}

}  // namespace apc
