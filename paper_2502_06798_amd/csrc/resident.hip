// Resident-aware fallback and the per-batch level histogram.
//
// k_resident_best: one wavefront per query; lane j looks up the residency of
// neighbour j (j < k) and a ballot picks the first resident one, i.e. the
// best, since the lists are ordered best first.  k_level_histogram: one block;
// each wavefront counts its queries per level with one ballot per level
// (lane l keeps level l's count), then adds the counts into LDS.
#include "apc_internal.h"

namespace apc {
namespace {

constexpr int RB_WAVES = 4;

__global__ __launch_bounds__(RB_WAVES * 64) void k_resident_best(const int32_t* __restrict__ slot_of_entry,
                                                                 int64_t n_entries, int64_t n_slots,
                                                                 const float* __restrict__ top_score,
                                                                 const int32_t* __restrict__ top_idx, int32_t ld,
                                                                 int32_t k, int32_t b, float* __restrict__ out_score,
                                                                 int32_t* __restrict__ out_idx)
{
    const int lane = threadIdx.x & 63;
    const int64_t q = (int64_t)blockIdx.x * RB_WAVES + (threadIdx.x >> 6);
    if (q >= b) return;                                   // uniform per wavefront
    bool res = false;
    int32_t e = -1;
    float s = 0.f;
    if (lane < k) {
        e = top_idx[q * ld + lane];
        s = top_score[q * ld + lane];
        if (e >= 0 && e < n_entries) {
            const int64_t slot = slot_of_entry ? (int64_t)slot_of_entry[e] : (int64_t)e;
            res = slot >= 0 && slot < n_slots;
        }
    }
    const uint64_t m = __ballot(res);
    const int j = m ? __builtin_ctzll(m) : 0;
    const int32_t ej = __shfl(e, j);
    const float sj = __shfl(s, j);
    if (lane == 0) {
        out_idx[q] = m ? ej : -1;
        out_score[q] = m ? sj : __builtin_nanf("");
    }
}

constexpr int LH_NT = 1024;

__global__ __launch_bounds__(LH_NT) void k_level_histogram(const int32_t* __restrict__ level, int32_t b, int32_t L,
                                                           int32_t* __restrict__ hist)
{
    __shared__ int h[APC_MAX_LEVELS + 1];
    const int tid = threadIdx.x, lane = tid & 63;
    if (tid <= L) h[tid] = 0;
    __syncthreads();
    int mine = 0;                                         // lane l: this wavefront's count of level l
    for (int base = 0; base < b; base += LH_NT) {
        const int q = base + tid;
        const int v = q < b ? level[q] : -1;
        for (int p = 0; p <= L; ++p) {
            const int c = __popcll(__ballot(v == p));
            if (lane == p) mine += c;
        }
    }
    if (lane <= L && mine) atomicAdd(&h[lane], mine);
    __syncthreads();
    if (tid <= L) hist[tid] = h[tid];
}

}  // namespace

hipError_t launch_resident_best(const int32_t* slot_of_entry, int64_t n_entries, int64_t n_slots,
                                const float* top_score, const int32_t* top_idx, int32_t ld, int32_t k, int32_t b,
                                float* out_score, int32_t* out_idx, hipStream_t s)
{
    if (b <= 0) return hipSuccess;
    const unsigned grid = (unsigned)((b + RB_WAVES - 1) / RB_WAVES);
    k_resident_best<<<grid, RB_WAVES * 64, 0, s>>>(slot_of_entry, n_entries, n_slots, top_score, top_idx, ld, k,
                                                   b, out_score, out_idx);
    return hipGetLastError();
}

hipError_t launch_level_histogram(const int32_t* level, int32_t b, int32_t L, int32_t* hist, hipStream_t s)
{
    k_level_histogram<<<1, LH_NT, 0, s>>>(level, b, L, hist);
    return hipGetLastError();
}

}  // namespace apc
