// Merge of the top-k lists of row shards of a cache (the step after the
// exchange of partial lists when the cache is split over devices): one
// wavefront per query, lane s owning the head of shard s's list.  Each round
// takes the wavefront maximum of the heads' keys, (score desc, global entry
// asc) packed into 64 bits, and the owning lane advances; the later loads of a
// list hit the cache lines its first load brought in.
#include "apc_internal.h"

namespace apc {
namespace {

constexpr int MS_WAVES = 4;

// order-preserving key; 0 is below every candidate (an empty head)
__device__ inline uint64_t shard_key(float s, int32_t e)
{
    const uint32_t u = __float_as_uint(s + 0.0f);            // -0 -> +0: equal scores
    const uint32_t o = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
    return ((uint64_t)o << 32) | (uint32_t)~(uint32_t)e;
}

// max with the key of the lane a DPP control names (own key where it names
// none or the row is masked off)
template <int CTRL, int ROWS>
__device__ inline uint64_t dpp_max(uint64_t v)
{
    const int lo = (int)(uint32_t)v, hi = (int)(uint32_t)(v >> 32);
    const uint64_t o = ((uint64_t)(uint32_t)__builtin_amdgcn_update_dpp(hi, hi, CTRL, ROWS, 0xf, false) << 32) |
                       (uint32_t)__builtin_amdgcn_update_dpp(lo, lo, CTRL, ROWS, 0xf, false);
    return o > v ? o : v;
}

// largest key of the wavefront: within quads, half rows and rows by
// permutes and mirrors, then across rows by the broadcasts of lanes 15 and
// 31; lane 63 ends with the maximum, read back as a scalar
__device__ inline uint64_t wave_max_u64(uint64_t v)
{
    v = dpp_max<0xB1, 0xf>(v);       // quad_perm [1, 0, 3, 2]
    v = dpp_max<0x4E, 0xf>(v);       // quad_perm [2, 3, 0, 1]
    v = dpp_max<0x141, 0xf>(v);      // row_half_mirror
    v = dpp_max<0x140, 0xf>(v);      // row_mirror
    v = dpp_max<0x142, 0xa>(v);      // row_bcast:15 into rows 1 and 3
    v = dpp_max<0x143, 0xc>(v);      // row_bcast:31 into rows 2 and 3
    const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)v, 63);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(v >> 32), 63);
    return ((uint64_t)hi << 32) | lo;
}

__global__ __launch_bounds__(MS_WAVES * 64) void k_merge_shards(const float* __restrict__ sc,
                                                                const int32_t* __restrict__ ix, int32_t g,
                                                                int32_t b, int32_t kin, const ShardOffsets off,
                                                                int32_t k, float* __restrict__ out_s,
                                                                int32_t* __restrict__ out_i)
{
    const int lane = threadIdx.x & 63;
    const int64_t q = (int64_t)blockIdx.x * MS_WAVES + (threadIdx.x >> 6);
    if (q >= b) return;                                       // uniform per wavefront
    const int64_t base = ((int64_t)lane * b + q) * kin;       // shard `lane`'s list of query q
    const int32_t o = lane < g ? off.v[lane] : 0;
    int head = 0;
    float hs = 0.f;
    int32_t he = 0;
    uint64_t key = 0;
    auto load = [&]() {
        key = 0;
        while (lane < g && head < kin) {                      // skip non-candidates
            hs = sc[base + head];
            const int32_t e = ix[base + head];
            // the global entry number, in 64 bits: one that does not fit below
            // 2^31 - 1 (the largest cache a handle takes) is not a candidate
            const int64_t ge = (int64_t)e + o;
            if (e >= 0 && hs == hs && ge < INT32_MAX) {
                he = (int32_t)ge;
                key = shard_key(hs, he);
                break;
            }
            ++head;
        }
    };
    load();
    for (int p = 0; p < k; ++p) {
        const uint64_t m = wave_max_u64(key);
        const bool mine = m != 0 && key == m;
        const uint64_t who = __ballot(mine);
        const int wl = who ? __builtin_ctzll(who) : 0;
        const float ws = __shfl(hs, wl);
        const int32_t we = __shfl(he, wl);
        if (lane == 0) {
            out_s[q * k + p] = who ? ws : __builtin_nanf("");
            out_i[q * k + p] = who ? we : -1;
        }
        if (mine) {
            ++head;
            load();
        }
    }
}

}  // namespace

hipError_t launch_merge_shards(const float* scores, const int32_t* idx, int32_t g, int32_t b, int32_t kin,
                               const ShardOffsets& off, int32_t k, float* out_s, int32_t* out_i, hipStream_t s)
{
    if (b <= 0) return hipSuccess;
    const unsigned grid = (unsigned)((b + MS_WAVES - 1) / MS_WAVES);
    k_merge_shards<<<grid, MS_WAVES * 64, 0, s>>>(scores, idx, g, b, kin, off, k, out_s, out_i);
    return hipGetLastError();
}

}  // namespace apc
