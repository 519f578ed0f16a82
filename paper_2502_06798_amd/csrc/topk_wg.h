// Workgroup-level exact top-k of a stream of (score, entry) pairs per query,
// and the per-type MFMA fragments shared by the similarity kernels.
//
// State per query (in LDS): a sorted list of the k best pairs so far (two
// copies: a merge writes the other one), an admission threshold, and a small
// buffer of candidates.  Lanes append pairs that beat the threshold; a merge
// round then gives every element of (list U candidates) its rank by counting
// the elements ahead of it in the order (score desc, entry asc), in parallel
// over all threads, and writes the k best to the other copy.  Candidates that
// do not fit in the buffer stay pending in their lane and are retried after
// the threshold has risen.  A pair is dropped only if k pairs that beat it
// have been seen, so the final list is the exact top-k of everything
// offered, whatever the order of arrival.
#pragma once

#include "apc_internal.h"

namespace apc {

typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef int i32x8 __attribute__((ext_vector_type(8)));

constexpr int IDX_NONE = 0x7fffffff;

__device__ inline float neg_inf() { return -__builtin_huge_valf(); }
__device__ inline float qnan() { return __int_as_float(0x7fc00000); }

// (sa, ia) comes before (sb, ib) in the order score desc, index asc
__device__ inline bool before(float sa, int ia, float sb, int ib)
{
    return sa > sb || (sa == sb && ia < ib);
}

__device__ inline float clamp1(float s) { return __builtin_fminf(__builtin_fmaxf(s, -1.f), 1.f); }

// ---- decoding (row norms) ----------------------------------------------------
__device__ inline float dec_e4m3(uint32_t c)
{
    // selects only (no branches): this runs on hundreds of codes per lane
    const uint32_t e = (c >> 3) & 15u, m = c & 7u;
    const float sub = (float)m * 0.001953125f;                             // m/8 * 2^-6
    const float nrm = __uint_as_float(((e + 120u) << 23) | (m << 20));     // (1 + m/8) * 2^(e - 7)
    float v = e == 0u ? sub : nrm;
    v = (c & 0x80u) ? -v : v;
    return (c & 0x7fu) == 0x7fu ? qnan() : v;
}

__device__ inline float dec_bf16(uint32_t h) { return __uint_as_float(h << 16); }

__device__ inline float dec_f16(uint32_t h)
{
    _Float16 x;
    uint16_t b = (uint16_t)h;
    __builtin_memcpy(&x, &b, 2);
    return (float)x;
}

// sum of squares of the elements packed in 16 bytes; bad |= any non-finite
template <int DT>
__device__ inline void sumsq16(const uint4 v, float& ss, bool& bad)
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
            for (int hh = 0; hh < 2; ++hh) {
                uint32_t c = (w[j] >> (16 * hh)) & 0xffffu;
                float x = DT == APC_F16 ? dec_f16(c) : dec_bf16(c);
                bad |= !__builtin_isfinite(x);
                ss = fmaf(x, x, ss);
            }
        } else {
#pragma unroll
            for (int hh = 0; hh < 4; ++hh) {
                float x = dec_e4m3((w[j] >> (8 * hh)) & 0xffu);
                bad |= !__builtin_isfinite(x);
                ss = fmaf(x, x, ss);
            }
        }
    }
}

// ---- MFMA over one 128-byte chunk of d ---------------------------------------
// 32x32 output block, entries = rows (A), queries = columns (B).  Lane l
// supplies row l % 32; half h = l / 32 supplies bytes [64h, 64h + 64) of the
// chunk for both operands (any lane -> k mapping works as long as A and B
// share it).  `a` holds the lane's 64 bytes of its entry row, `qb` points at
// the lane's 64 bytes of its query row in LDS.
template <int DT> struct ChunkMma;

template <> struct ChunkMma<APC_F16> {
    __device__ static void run(f32x16& c, const uint4 (&a)[4], const uint8_t* qb)
    {
#pragma unroll
        for (int s = 0; s < 4; ++s) {
            const f16x8 b = *reinterpret_cast<const f16x8*>(qb + 16 * s);
            c = __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(f16x8, a[s]), b, c, 0, 0, 0);
        }
    }
};

template <> struct ChunkMma<APC_BF16> {
    __device__ static void run(f32x16& c, const uint4 (&a)[4], const uint8_t* qb)
    {
#pragma unroll
        for (int s = 0; s < 4; ++s) {
            const bf16x8 b = *reinterpret_cast<const bf16x8*>(qb + 16 * s);
            c = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a[s]), b, c, 0, 0, 0);
        }
    }
};

template <> struct ChunkMma<APC_E4M3> {
    __device__ static void run(f32x16& c, const uint4 (&a)[4], const uint8_t* qb)
    {
#pragma unroll
        for (int s = 0; s < 2; ++s) {
            const i32x8 b = *reinterpret_cast<const i32x8*>(qb + 32 * s);
            const i32x8 av = {(int)a[2 * s].x, (int)a[2 * s].y, (int)a[2 * s].z, (int)a[2 * s].w,
                              (int)a[2 * s + 1].x, (int)a[2 * s + 1].y, (int)a[2 * s + 1].z,
                              (int)a[2 * s + 1].w};
            c = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(av, b, c, 0, 0, 0, 0, 0, 0);
        }
    }
};

template <> struct ChunkMma<APC_F32> {
    __device__ static void run(f32x16& c, const uint4 (&a)[4], const uint8_t* qb)
    {
#pragma unroll
        for (int s = 0; s < 4; ++s) {
            const float4 b = *reinterpret_cast<const float4*>(qb + 16 * s);
            c = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a[s].x), b.x, c, 0, 0, 0);
            c = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a[s].y), b.y, c, 0, 0, 0);
            c = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a[s].z), b.z, c, 0, 0, 0);
            c = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a[s].w), b.w, c, 0, 0, 0);
        }
    }
};

// ---- workgroup top-k state ---------------------------------------------------
template <int BQ, int KMAX, int NCAND>
struct TopkLds {
    float list_s[2][KMAX * BQ];   // [copy][p * BQ + q], sorted desc, sentinel-padded
    int list_i[2][KMAX * BQ];
    float cand_s[BQ * NCAND];
    int cand_i[BQ * NCAND];
    float thr_s[BQ];              // admission threshold: pairs must come before it
    int thr_i[BQ];
    int cnt[BQ];
    int cur[BQ];
};

template <int BQ, int KMAX, int NCAND, int NT>
__device__ inline void topk_init(TopkLds<BQ, KMAX, NCAND>& st, int tid)
{
    for (int i = tid; i < KMAX * BQ; i += NT) {
        st.list_s[0][i] = neg_inf();
        st.list_i[0][i] = IDX_NONE;
    }
    for (int q = tid; q < BQ; q += NT) {
        st.thr_s[q] = neg_inf();
        st.thr_i[q] = IDX_NONE;
        st.cnt[q] = 0;
        st.cur[q] = 0;
    }
}

// Try to append one pair; returns true when it is settled (stored or below the threshold).
template <int BQ, int KMAX, int NCAND>
__device__ inline bool topk_offer(TopkLds<BQ, KMAX, NCAND>& st, int q, float s, int e)
{
    if (!before(s, e, st.thr_s[q], st.thr_i[q])) return true;
    const int pos = atomicAdd(&st.cnt[q], 1);
    if (pos >= NCAND) return false;
    st.cand_s[q * NCAND + pos] = s;
    st.cand_i[q * NCAND + pos] = e;
    return true;
}

// Merge round, part 1 (after a barrier): rank every element of list U candidates
// of each query that has candidates, and write the k best to the other copy.
template <int BQ, int KMAX, int NCAND, int NT>
__device__ inline void topk_rank(TopkLds<BQ, KMAX, NCAND>& st, int k, int tid)
{
    constexpr int PER = KMAX + NCAND;
    for (int task = tid; task < BQ * PER; task += NT) {
        const int q = task / PER, j = task % PER;
        const int c0 = st.cnt[q];
        if (c0 == 0) continue;
        const int c = c0 < NCAND ? c0 : NCAND;
        const int cur = st.cur[q];
        const float* ls = st.list_s[cur];
        const int* li = st.list_i[cur];
        const float* cs = st.cand_s + q * NCAND;
        const int* ci = st.cand_i + q * NCAND;
        float s;
        int e, rank;
        if (j < KMAX) {
            if (j >= k) continue;
            s = ls[j * BQ + q];
            e = li[j * BQ + q];
            rank = j;
            for (int x = 0; x < c; ++x) rank += before(cs[x], ci[x], s, e);
        } else {
            const int x0 = j - KMAX;
            if (x0 >= c) continue;
            s = cs[x0];
            e = ci[x0];
            rank = 0;
            for (int p = 0; p < k; ++p) rank += before(ls[p * BQ + q], li[p * BQ + q], s, e);
            for (int x = 0; x < c; ++x) rank += before(cs[x], ci[x], s, e);
        }
        if (rank < k) {
            st.list_s[cur ^ 1][rank * BQ + q] = s;
            st.list_i[cur ^ 1][rank * BQ + q] = e;
        }
    }
}

// Merge round, part 2 (after a barrier): switch copies, raise thresholds, empty buffers.
template <int BQ, int KMAX, int NCAND, int NT>
__device__ inline void topk_finish(TopkLds<BQ, KMAX, NCAND>& st, int k, int tid)
{
    for (int q = tid; q < BQ; q += NT) {
        if (st.cnt[q] == 0) continue;
        const int cur = st.cur[q] ^ 1;
        st.cur[q] = cur;
        const float s = st.list_s[cur][(k - 1) * BQ + q];
        const int e = st.list_i[cur][(k - 1) * BQ + q];
        if (before(s, e, st.thr_s[q], st.thr_i[q])) {
            st.thr_s[q] = s;
            st.thr_i[q] = e;
        }
        st.cnt[q] = 0;
    }
}

}  // namespace apc
