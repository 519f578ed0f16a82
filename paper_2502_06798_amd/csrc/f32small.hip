// Similarity + top-k for float32 caches of at most 16,384 rows (the batch's
// nearest cached prompts, Approach / Query Dispatcher).
//
// A small float32 cache gives each CU only a block or two of 32 rows, and one
// wavefront working through all of d in one accumulation chain is latency
// bound.  Here a workgroup takes one 32-row block against a tile of 16
// queries, and its NW wavefronts (eight when d is a multiple of 128, else
// four) take equal parts of d with 16x16x4 float32 MFMAs (two row tiles of
// 16); the partial sums meet in LDS.  A lane of wavefront w supplies, at
// step (t, j), row i = lane % 16 and column w d/NW + 16 t + 4 (lane / 16) + j
// of both operands, so the two operands see the same column for every
// product and each lane reads 16 contiguous bytes of its row per step.  Every query's 32 scores then give the block's
// partial list (k best, sorted by score desc then entry asc, each pair placed
// by its rank; rows past the cache are -inf), which k_topk_merge merges over
// the blocks.
#include <type_traits>

#include "apc_internal.h"

namespace apc {
namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int FS_QT = 16;      // queries per tile
constexpr int FS_ROWS = 32;    // cache rows per workgroup
constexpr int FS_NONE = 0x7fffffff;

__device__ inline float fs_clamp1(float x) { return __builtin_fminf(__builtin_fmaxf(x, -1.0f), 1.0f); }

template <int FS_NW>
__global__ __launch_bounds__(FS_NW * 64) void k_f32s(const float* __restrict__ emb, const float* __restrict__ fe,
                                                    int64_t n, int32_t d, const float* __restrict__ q,
                                                    const float* __restrict__ fq, int32_t b, int32_t k, int splits,
                                                    float* __restrict__ part_s, int* __restrict__ part_i)
{
    __shared__ f32x4 red[FS_NW][2][64];
    __shared__ float sc[FS_QT][FS_ROWS + 1];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int i16 = lane & 15, kq = lane >> 4;
    const int split = blockIdx.x;
    const int64_t r0 = (int64_t)split * FS_ROWS, q0 = (int64_t)blockIdx.y * FS_QT;

    // this lane's two rows and query (clamped into the arrays; their scores
    // are masked below)
    const int64_t ra = r0 + i16 < n ? r0 + i16 : n - 1;
    const int64_t rb = r0 + 16 + i16 < n ? r0 + 16 + i16 : n - 1;
    const int64_t qq = q0 + i16 < b ? q0 + i16 : b - 1;
    const int dw = d / FS_NW, c0 = wave * dw + 4 * kq;
    const float* pa = emb + ra * d + c0;
    const float* pb = emb + rb * d + c0;
    const float* pq = q + qq * d + c0;
    f32x4 acc0 = {0.f, 0.f, 0.f, 0.f}, acc1 = {0.f, 0.f, 0.f, 0.f};
    // steps of 16 columns, in chunks of CH, two chunk buffers: the next
    // chunk's loads are in flight while a chunk's MFMAs run
    constexpr int CH = 4;
    const int nt = dw / 16;
    float4 a[2][CH], c[2][CH], y[2][CH];
    auto load = [&](auto bc, int t0) __attribute__((always_inline)) {
        constexpr int bf = decltype(bc)::value;
#pragma unroll
        for (int j = 0; j < CH; ++j)
            if (t0 + j < nt) {
                a[bf][j] = *reinterpret_cast<const float4*>(pa + 16 * (t0 + j));
                c[bf][j] = *reinterpret_cast<const float4*>(pb + 16 * (t0 + j));
                y[bf][j] = *reinterpret_cast<const float4*>(pq + 16 * (t0 + j));
            }
    };
    auto mma = [&](auto bc, int t0) __attribute__((always_inline)) {
        constexpr int bf = decltype(bc)::value;
#pragma unroll
        for (int j = 0; j < CH; ++j)
            if (t0 + j < nt) {
                const float4 x0 = a[bf][j], x1 = c[bf][j], yq = y[bf][j];
                acc0 = __builtin_amdgcn_mfma_f32_16x16x4f32(x0.x, yq.x, acc0, 0, 0, 0);
                acc1 = __builtin_amdgcn_mfma_f32_16x16x4f32(x1.x, yq.x, acc1, 0, 0, 0);
                acc0 = __builtin_amdgcn_mfma_f32_16x16x4f32(x0.y, yq.y, acc0, 0, 0, 0);
                acc1 = __builtin_amdgcn_mfma_f32_16x16x4f32(x1.y, yq.y, acc1, 0, 0, 0);
                acc0 = __builtin_amdgcn_mfma_f32_16x16x4f32(x0.z, yq.z, acc0, 0, 0, 0);
                acc1 = __builtin_amdgcn_mfma_f32_16x16x4f32(x1.z, yq.z, acc1, 0, 0, 0);
                acc0 = __builtin_amdgcn_mfma_f32_16x16x4f32(x0.w, yq.w, acc0, 0, 0, 0);
                acc1 = __builtin_amdgcn_mfma_f32_16x16x4f32(x1.w, yq.w, acc1, 0, 0, 0);
            }
    };
    using B0 = std::integral_constant<int, 0>;
    using B1 = std::integral_constant<int, 1>;
    load(B0{}, 0);
    for (int t0 = 0; t0 < nt; t0 += 2 * CH) {
        load(B1{}, t0 + CH);
        mma(B0{}, t0);
        load(B0{}, t0 + 2 * CH);
        mma(B1{}, t0 + CH);
    }
    red[wave][0][lane] = acc0;
    red[wave][1][lane] = acc1;
    __syncthreads();

    // wavefront 0: the parts of d summed in a fixed order, times the
    // factors, clamped.  Lane l holds rows 4 (l / 16) + v of each row tile
    // against query l % 16.
    if (wave == 0) {
        const int64_t qg = q0 + i16;
        const float f = qg < b ? fq[qg] : 0.f;
#pragma unroll
        for (int tl = 0; tl < 2; ++tl) {
            f32x4 s = red[0][tl][lane];
#pragma unroll
            for (int w = 1; w < FS_NW; ++w) s += red[w][tl][lane];
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int rl = 16 * tl + 4 * kq + v;
                const int64_t r = r0 + rl;
                sc[i16][rl] = r < n ? fs_clamp1(s[v] * fe[r] * f) : -__builtin_huge_valf();
            }
        }
    }
    __syncthreads();

    // each (query, row) pair finds its rank among the query's 32 scores
    // (score desc, row asc); the pairs of rank below k are the partial list
    for (int e = tid; e < FS_QT * FS_ROWS; e += FS_NW * 64) {
        const int qi = e / FS_ROWS, rl = e % FS_ROWS;
        const float x = sc[qi][rl];
        int rank = 0;
#pragma unroll 8
        for (int r2 = 0; r2 < FS_ROWS; ++r2) {
            const float z = sc[qi][r2];
            rank += z > x || (z == x && r2 < rl);
        }
        if (rank < k) {
            const int64_t o = ((q0 + qi) * splits + split) * k + rank;
            const bool real = r0 + rl < n;
            part_s[o] = real ? x : -__builtin_huge_valf();
            part_i[o] = real ? (int)(r0 + rl) : FS_NONE;
        }
    }
}

}  // namespace

bool f32s_fits(int dt, int64_t n, int32_t d, int32_t b, int32_t k)
{
    return dt == APC_F32 && d >= 64 && d % 64 == 0 && k >= 1 && k <= FS_ROWS && n >= 1 &&
           (n + FS_ROWS - 1) / FS_ROWS <= 512 && b >= 1 && b <= 256;
}

int f32s_queries() { return FS_QT; }
int f32s_rows() { return FS_ROWS; }

hipError_t launch_f32s(const MatchPlan& p, int64_t n, int32_t d, const void* emb, const float* fe, const void* q,
                       const float* fq, int32_t b, int32_t k, float* ps, int* pi, hipStream_t s)
{
    const dim3 grid((unsigned)p.splits, (unsigned)p.qtiles);
    const float* e = static_cast<const float*>(emb);
    const float* qf = static_cast<const float*>(q);
    if (d % 128 == 0) k_f32s<8><<<grid, dim3(8 * 64), 0, s>>>(e, fe, n, d, qf, fq, b, k, p.splits, ps, pi);
    else k_f32s<4><<<grid, dim3(4 * 64), 0, s>>>(e, fe, n, d, qf, fq, b, k, p.splits, ps, pi);
    return hipGetLastError();
}

}  // namespace apc
