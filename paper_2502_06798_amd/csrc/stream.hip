// Streaming similarity + top-k for small query batches (the HBM-bound regime).
//
// Each workgroup keeps a tile of BQ queries resident in LDS for its whole
// life and streams its range of cache entries straight from HBM into MFMA
// registers: lane l of a wavefront loads 64 contiguous bytes of entry row
// (l % 32) per 128-byte chunk of d (half l / 32 takes the upper 64 bytes),
// four chunks in flight, and the same bytes of its query row come from LDS
// one chunk ahead.  Loads are unconditional (rows past the end read the last
// row and are ignored later; rows are whole 128-byte chunks) so the compiler
// waits on exactly the chunk it needs.  Entries are the MFMA
// rows (32-entry blocks), queries the columns, so one query fragment feeds
// two entry blocks.  Four wavefronts (one per SIMD, 512 registers each) take
// disjoint 64-entry slices per round.
//
// Epilogue per round (all in registers until something can enter a top-k):
// per query block each lane takes maxima of its products acc * f_e over four
// groups of 8 entries; since scaling by f_q > 0 and clamping are monotone,
// clamp(max * f_q) is exactly the best score of a group, and only lanes whose
// best beats the query's threshold compute individual scores.  On the first
// round the k-th largest of the 32 group maxima of each query (32 disjoint
// entry subsets) gives the starting threshold, so the workgroup never floods
// its candidate buffers.  The exact top-k bookkeeping is in topk_wg.h.
#include <type_traits>

#include "topk_wg.h"

namespace apc {
namespace {

constexpr int NCAND_S = 32;
constexpr int STREAM_WAVES = 4;    // one wavefront per SIMD

constexpr int NSPL = 4;             // entry groups (of 8) per lane and query block

template <int BQ, int QB, int KMAX, int NW>
struct StreamCfg {
    static constexpr int NT = NW * 64;
    static constexpr int MQ = BQ / 32;
    static constexpr int QSTRIDE = QB + 16;     // 16 consecutive rows start on distinct bank quads
    static constexpr int NSUB = 2 * NW * NSPL;  // disjoint entry subsets per query per round
    struct Smem {
        uint8_t q[BQ * QSTRIDE];
        TopkLds<BQ, KMAX, NCAND_S> st;
        float fq[BQ];
        float bmax[BQ * NSUB];
    };
};

// one 128-byte chunk of d: a = the lane's 64 bytes of each entry row, b = its
// 64 bytes of each query row
template <int DT, int MQ, int ME>
__device__ inline void mma_chunk(f32x16 (&acc)[MQ][2], const uint4 (&a)[ME][4], const uint4 (&b)[MQ][4])
{
#pragma unroll
    for (int mq = 0; mq < MQ; ++mq) {
        if constexpr (DT == APC_F16 || DT == APC_BF16) {
            typedef typename std::conditional<DT == APC_F16, f16x8, bf16x8>::type V;
#pragma unroll
            for (int s = 0; s < 4; ++s)
#pragma unroll
                for (int me = 0; me < ME; ++me) {
                    if constexpr (DT == APC_F16)
                        acc[mq][me] = __builtin_amdgcn_mfma_f32_32x32x16_f16(
                            __builtin_bit_cast(V, a[me][s]), __builtin_bit_cast(V, b[mq][s]), acc[mq][me], 0, 0, 0);
                    else
                        acc[mq][me] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                            __builtin_bit_cast(V, a[me][s]), __builtin_bit_cast(V, b[mq][s]), acc[mq][me], 0, 0, 0);
                }
        } else if constexpr (DT == APC_E4M3) {
#pragma unroll
            for (int s = 0; s < 2; ++s) {
                const uint4 blo = b[mq][2 * s], bhi = b[mq][2 * s + 1];
                const i32x8 bv = {(int)blo.x, (int)blo.y, (int)blo.z, (int)blo.w,
                                  (int)bhi.x, (int)bhi.y, (int)bhi.z, (int)bhi.w};
#pragma unroll
                for (int me = 0; me < ME; ++me) {
                    const uint4 lo = a[me][2 * s], hi = a[me][2 * s + 1];
                    const i32x8 av = {(int)lo.x, (int)lo.y, (int)lo.z, (int)lo.w,
                                      (int)hi.x, (int)hi.y, (int)hi.z, (int)hi.w};
                    acc[mq][me] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(av, bv, acc[mq][me], 0, 0, 0, 0, 0, 0);
                }
            }
        } else {
#pragma unroll
            for (int s = 0; s < 4; ++s)
#pragma unroll
                for (int me = 0; me < ME; ++me) {
                    const uint4 x = a[me][s], y = b[mq][s];
                    acc[mq][me] = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(x.x), __uint_as_float(y.x), acc[mq][me], 0, 0, 0);
                    acc[mq][me] = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(x.y), __uint_as_float(y.y), acc[mq][me], 0, 0, 0);
                    acc[mq][me] = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(x.z), __uint_as_float(y.z), acc[mq][me], 0, 0, 0);
                    acc[mq][me] = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(x.w), __uint_as_float(y.w), acc[mq][me], 0, 0, 0);
                }
        }
    }
}

// chunks of d in flight per wavefront: even, and dividing the chunks of a row
// so the look-ahead runs on into the next round with the same buffer slots
template <int DT> struct StreamNB { static constexpr int NB = DT == APC_E4M3 ? 6 : 4; };

template <int DT, int BQ, int QB, int KMAX, int NW>
__global__ __launch_bounds__(NW * 64) void k_stream(
    const uint8_t* __restrict__ emb, const float* __restrict__ fe, int64_t n,
    const uint8_t* __restrict__ qry, const float* __restrict__ q_scale, int32_t b,
    int64_t row_bytes, int32_t k, int splits, int64_t b_pad,
    float* __restrict__ fq_out, float* __restrict__ part_s, int* __restrict__ part_i)
{
    typedef StreamCfg<BQ, QB, KMAX, NW> C;
    constexpr int MQ = C::MQ, NT = C::NT, QS = C::QSTRIDE, NB = StreamNB<DT>::NB;
    constexpr bool REG_LISTS = KMAX <= 16;      // lists in registers of one owner thread per query
    constexpr int KR = REG_LISTS ? KMAX : 1;
    __shared__ typename C::Smem sm;
    auto& st = sm.st;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, h = lane >> 5, r32 = lane & 31;
    const int split = blockIdx.x;
    const int64_t q0 = (int64_t)blockIdx.y * BQ;

    // ---- schedule: rounds of 2 blocks of 32 entries per wavefront ----
    const int64_t nblk = (n + 31) / 32;
    const int64_t b_begin = nblk * split / splits, b_end = nblk * (split + 1) / splits;
    const int64_t rounds = (b_end - b_begin + 2 * NW - 1) / (2 * NW);
    // blocks of round rd for this wavefront; the last round spreads its blocks
    auto blocks_of = [&](int64_t rd, int64_t (&blk)[2], int& me_n) {
        const int64_t base = b_begin + rd * 2 * NW, rem = b_end - base;
        if (rem >= 2 * NW) {
            blk[0] = base + 2 * wave;
            blk[1] = blk[0] + 1;
            me_n = 2;
        } else {
            blk[0] = base + wave;
            blk[1] = base + wave + NW;
            me_n = rd < rounds ? (wave < rem) + (wave + NW < rem) : 0;
        }
    };
    // row pointers of the lane (blocks outside the range re-read the range's
    // first rows: in cache, and their scores are never used)
    auto rows_of = [&](const int64_t (&blk)[2], int me_n, const uint8_t* (&rp)[2]) {
#pragma unroll
        for (int me = 0; me < 2; ++me) {
            int64_t e = blk[me] * 32 + r32;
            if (!(me < me_n && e < n)) e = b_begin * 32 + r32 < n ? b_begin * 32 + r32 : n - 1;
            rp[me] = emb + e * row_bytes + h * 64;
        }
    };
    auto load_e = [&](const uint8_t* const (&rp)[2], int c, uint4 (&dst)[2][4]) {
#pragma unroll
        for (int me = 0; me < 2; ++me)
#pragma unroll
            for (int u = 0; u < 4; ++u)
                dst[me][u] = *reinterpret_cast<const uint4*>(rp[me] + (int64_t)c * 128 + 16 * u);
    };

    // the first chunks of the stream go out before anything else
    uint4 ea[NB][2][4];
    int64_t blk[2];
    int me_n;
    const uint8_t* rp_cur[2];
    blocks_of(0, blk, me_n);
    rows_of(blk, me_n, rp_cur);
#pragma unroll
    for (int j = 0; j < NB - 1; ++j) load_e(rp_cur, j, ea[j]);

    // query tile -> LDS (zero padded): all loads in flight, then the stores
    const int nc16 = (int)(row_bytes / 16);
    {
        constexpr int NQL = BQ * (QB / 16) / NT;
        static_assert(BQ * (QB / 16) % NT == 0, "query tile must split evenly");
        uint4 v[NQL];
#pragma unroll
        for (int j = 0; j < NQL; ++j) {
            const int i = tid + j * NT, r = i / (QB / 16), c = i % (QB / 16);
            v[j] = (c < nc16 && q0 + r < b) ? *reinterpret_cast<const uint4*>(qry + (q0 + r) * row_bytes + c * 16)
                                           : make_uint4(0, 0, 0, 0);
        }
#pragma unroll
        for (int j = 0; j < NQL; ++j) {
            const int i = tid + j * NT, r = i / (QB / 16), c = i % (QB / 16);
            *reinterpret_cast<uint4*>(sm.q + r * QS + c * 16) = v[j];
        }
    }
    topk_init<BQ, KMAX, NCAND_S, NT>(st, tid);
    float ls[KR];
    int li[KR];
#pragma unroll
    for (int p = 0; p < KR; ++p) {
        ls[p] = neg_inf();
        li[p] = IDX_NONE;
    }
    __syncthreads();

    // query factors (NaN marks a row that cannot be matched)
    for (int r = wave; r < BQ; r += NW) {
        float ss = 0.f;
        bool bad = false;
        for (int c = lane; c < nc16; c += 64) sumsq16<DT>(*reinterpret_cast<const uint4*>(sm.q + r * QS + c * 16), ss, bad);
#pragma unroll
        for (int m = 32; m >= 1; m >>= 1) ss += __shfl_xor(ss, m, 64);
        bad = __any(bad);
        if (lane == 0) {
            const int64_t qg = q0 + r;
            float f = qnan();
            if (qg < b) {
                bool ok = !bad && __builtin_isfinite(ss) && ss > 0.f;
                if (q_scale) {
                    const float sc = q_scale[qg];
                    ok = ok && __builtin_isfinite(sc) && sc > 0.f;
                }
                if (ok) f = 1.0f / __builtin_sqrtf(ss);
                if (split == 0) fq_out[qg] = f;
            }
            sm.fq[r] = f;
        }
    }
    __syncthreads();

    const int nch = (int)(row_bytes / 128);      // a multiple of NB here
    const uint8_t* qrow = sm.q + r32 * QS + h * 64;
    uint4 qb[2][MQ][4];
    auto load_q = [&](int c, uint4 (&dst)[MQ][4]) {
#pragma unroll
        for (int mq = 0; mq < MQ; ++mq)
#pragma unroll
            for (int u = 0; u < 4; ++u)
                dst[mq][u] = *reinterpret_cast<const uint4*>(qrow + mq * 32 * QS + c * 128 + 16 * u);
    };
    load_q(0, qb[0]);

    for (int64_t rd = 0; rd < rounds; ++rd) {
        int64_t blk_nx[2];
        int me_nx;
        const uint8_t* rp_nx[2];
        blocks_of(rd + 1, blk_nx, me_nx);
        rows_of(blk_nx, me_nx, rp_nx);
        // entry factors of this round, consumed by the epilogue
        float4 fe4[2][4];
#pragma unroll
        for (int me = 0; me < 2; ++me)
#pragma unroll
            for (int g = 0; g < 4; ++g)
                fe4[me][g] = *reinterpret_cast<const float4*>(fe + (me < me_n ? blk[me] * 32 : 0) + 8 * g + 4 * h);

        f32x16 acc[MQ][2];
#pragma unroll
        for (int mq = 0; mq < MQ; ++mq)
#pragma unroll
            for (int me = 0; me < 2; ++me)
#pragma unroll
                for (int r = 0; r < 16; ++r) acc[mq][me][r] = 0.f;

        // one continuous stream: the look-ahead past this round's last chunk
        // loads the next round's first chunks into the same buffer slots
        for (int c0 = 0; c0 < nch; c0 += NB) {
#pragma unroll
            for (int j = 0; j < NB; ++j) {
                const int c = c0 + j;
                const int t = c + NB - 1;
                const bool here = t < nch;
                const uint8_t* rp[2] = {here ? rp_cur[0] : rp_nx[0], here ? rp_cur[1] : rp_nx[1]};
                __builtin_amdgcn_sched_barrier(0);
                load_e(rp, here ? t : t - nch, ea[(j + NB - 1) % NB]);
                load_q(c + 1 < nch ? c + 1 : 0, qb[(j + 1) & 1]);
                mma_chunk<DT, MQ, 2>(acc, ea[j], qb[j & 1]);
            }
        }
        __builtin_amdgcn_sched_barrier(0);

        // ---- epilogue ----
        // entry of score r of block me: blk*32 + 8*(r/4) + 4*h + r%4; valid below lim[me]
        int lim[2];
#pragma unroll
        for (int me = 0; me < 2; ++me) {
            const int64_t l = me < me_n ? n - (blk[me] * 32 + 4 * h) : 0;
            lim[me] = l > 64 ? 64 : (int)l;
        }
        float mx[MQ];                             // best score of the lane per query block
        float sub[MQ][NSPL];                      // ... and of each group of 8 entries
#pragma unroll
        for (int mq = 0; mq < MQ; ++mq) {
            const float f = sm.fq[mq * 32 + r32];
            float best = neg_inf();
#pragma unroll
            for (int gsp = 0; gsp < NSPL; ++gsp) {
                const int me = gsp >> 1, r0 = (gsp & 1) * 8;
                float m = neg_inf();
#pragma unroll
                for (int r = r0; r < r0 + 8; ++r) {
                    const float4 f4 = fe4[me][r >> 2];
                    const float fv = (r & 3) == 0 ? f4.x : (r & 3) == 1 ? f4.y : (r & 3) == 2 ? f4.z : f4.w;
                    const float v = acc[mq][me][r] * fv;
                    acc[mq][me][r] = v;
                    if (8 * (r >> 2) + (r & 3) < lim[me]) m = __builtin_fmaxf(m, v);
                }
                sub[mq][gsp] = (m == neg_inf() || !(f == f)) ? neg_inf() : clamp1(m * f);
                best = __builtin_fmaxf(best, sub[mq][gsp]);
            }
            mx[mq] = best;
        }
        if (rd == 0 && k <= C::NSUB) {
            // starting thresholds: k-th largest of the group maxima (disjoint subsets)
#pragma unroll
            for (int mq = 0; mq < MQ; ++mq)
#pragma unroll
                for (int gsp = 0; gsp < NSPL; ++gsp)
                    sm.bmax[(mq * 32 + r32) * C::NSUB + (wave * 2 + h) * NSPL + gsp] = sub[mq][gsp];
            __syncthreads();
            if (tid < BQ) {
                float v[C::NSUB];
#pragma unroll
                for (int i = 0; i < C::NSUB; ++i) v[i] = sm.bmax[tid * C::NSUB + i];
                float kth = neg_inf();
                for (int it = 0; it < k; ++it) {          // take the maximum out k times
                    float m = neg_inf();
#pragma unroll
                    for (int i = 0; i < C::NSUB; ++i) m = __builtin_fmaxf(m, v[i]);
                    bool gone = false;
#pragma unroll
                    for (int i = 0; i < C::NSUB; ++i) {
                        const bool hit = !gone && v[i] == m;
                        gone |= hit;
                        v[i] = hit ? neg_inf() : v[i];
                    }
                    kth = m;
                }
                if (kth > neg_inf()) {
                    st.thr_s[tid] = kth;
                    st.thr_i[tid] = IDX_NONE;            // admits every pair with score >= kth
                }
            }
            __syncthreads();
        }
        // exact scores only where a group maximum reaches the threshold; pairs that
        // pass go straight to the query's buffer, overflow stays pending
        uint64_t pend = 0;
        bool ovf = false;
#pragma unroll
        for (int mq = 0; mq < MQ; ++mq) {
            const int ql = mq * 32 + r32;
            const float ts = st.thr_s[ql];
            const int ti = st.thr_i[ql];
            if (mx[mq] >= ts && mx[mq] > neg_inf()) {
                const float f = sm.fq[ql];
#pragma unroll
                for (int me = 0; me < 2; ++me)
#pragma unroll
                    for (int r = 0; r < 16; ++r) {
                        const float sc = clamp1(acc[mq][me][r] * f);
                        acc[mq][me][r] = sc;
                        const int e = (int)(blk[me] * 32 + 8 * (r >> 2) + 4 * h + (r & 3));
                        if (8 * (r >> 2) + (r & 3) < lim[me] && before(sc, e, ts, ti)) {
                            const int pos = atomicAdd(&st.cnt[ql], 1);
                            if (pos < NCAND_S) {
                                st.cand_s[ql * NCAND_S + pos] = sc;
                                st.cand_i[ql * NCAND_S + pos] = e;
                            } else {
                                pend |= 1ull << ((mq * 2 + me) * 16 + r);
                                ovf = true;
                            }
                        }
                    }
            }
        }
        // merge rounds: the first merges this round's appends; after an overflow
        // each further pass merges the re-offered pairs
        bool again = __syncthreads_or(ovf);
        for (bool more = true; more;) {
            more = again;
            if constexpr (REG_LISTS) {
                if (tid < BQ && st.cnt[tid] > 0) {      // owner of query tid merges its buffer
                    int c = st.cnt[tid];
                    c = c < NCAND_S ? c : NCAND_S;
                    float ts = st.thr_s[tid];
                    int ti = st.thr_i[tid];
                    for (int x = 0; x < c; ++x) {
                        const float sv = st.cand_s[tid * NCAND_S + x];
                        const int ev = st.cand_i[tid * NCAND_S + x];
                        if (!before(sv, ev, ts, ti)) continue;
                        // the pair beats the k-th: shift lower entries down from k-1
                        bool placed = false;
#pragma unroll
                        for (int p = KR - 1; p >= 1; --p) {
                            if (p < k && !placed) {
                                const bool up = before(sv, ev, ls[p - 1], li[p - 1]);
                                ls[p] = up ? ls[p - 1] : sv;
                                li[p] = up ? li[p - 1] : ev;
                                placed = !up;
                            }
                        }
                        if (!placed) {
                            ls[0] = sv;
                            li[0] = ev;
                        }
                        float ks = neg_inf();
                        int ki = IDX_NONE;
#pragma unroll
                        for (int p = 0; p < KR; ++p)
                            if (p == k - 1) { ks = ls[p]; ki = li[p]; }
                        if (before(ks, ki, ts, ti)) { ts = ks; ti = ki; }
                    }
                    st.thr_s[tid] = ts;
                    st.thr_i[tid] = ti;
                    st.cnt[tid] = 0;
                }
            } else {
                topk_rank<BQ, KMAX, NCAND_S, NT>(st, k, tid);
                __syncthreads();
                topk_finish<BQ, KMAX, NCAND_S, NT>(st, k, tid);
            }
            if (!more) break;
            // rare: a buffer overflowed; offer the pending pairs again after the
            // merge, then merge what they stored (and repeat while anything is left)
            __syncthreads();
            if (pend) {
#pragma unroll
                for (int mq = 0; mq < MQ; ++mq)
#pragma unroll
                    for (int me = 0; me < 2; ++me)
#pragma unroll
                        for (int r = 0; r < 16; ++r) {
                            const int bit = (mq * 2 + me) * 16 + r;
                            if ((pend >> bit) & 1) {
                                const int e = (int)(blk[me] * 32 + 8 * (r >> 2) + 4 * h + (r & 3));
                                if (topk_offer(st, mq * 32 + r32, acc[mq][me][r], e)) pend &= ~(1ull << bit);
                            }
                        }
            }
            again = __syncthreads_or(pend != 0);
        }
        __syncthreads();

        blk[0] = blk_nx[0];
        blk[1] = blk_nx[1];
        me_n = me_nx;
        rp_cur[0] = rp_nx[0];
        rp_cur[1] = rp_nx[1];
    }

    if constexpr (REG_LISTS) {
        if (tid < BQ) {
            const int64_t o = (((int64_t)q0 + tid) * splits + split) * k;
#pragma unroll
            for (int p = 0; p < KR; ++p)
                if (p < k) {
                    part_s[o + p] = ls[p];
                    part_i[o + p] = li[p];
                }
        }
    } else {
        for (int i = tid; i < BQ * k; i += NT) {
            const int q = i / k, p = i % k;
            const int64_t o = (((int64_t)q0 + q) * splits + split) * k + p;
            part_s[o] = st.list_s[st.cur[q]][p * BQ + q];
            part_i[o] = st.list_i[st.cur[q]][p * BQ + q];
        }
    }
}

template <int DT, int BQ, int QB, int KMAX>
hipError_t run_stream(const MatchPlan& p, int64_t n, const void* emb, const float* fe, const void* q,
                      const float* q_scale, int32_t b, int64_t row_bytes, int32_t k, float* fq,
                      float* ps, int* pi, hipStream_t s)
{
    constexpr int NW = STREAM_WAVES;
    const dim3 grid(p.splits, p.qtiles), block(NW * 64);
    k_stream<DT, BQ, QB, KMAX, NW><<<grid, block, 0, s>>>(
        static_cast<const uint8_t*>(emb), fe, n, static_cast<const uint8_t*>(q), q_scale, b,
        row_bytes, k, p.splits, p.b_pad, fq, ps, pi);
    return hipGetLastError();
}

template <int DT>
hipError_t run_stream_dt(const MatchPlan& p, int64_t n, const void* emb, const float* fe, const void* q,
                         const float* q_scale, int32_t b, int64_t row_bytes, int32_t k, float* fq,
                         float* ps, int* pi, hipStream_t s)
{
    if constexpr (DT != APC_E4M3)                // e4m3 keeps six chunks in flight: 32-query tiles only
        if (p.kernel == KERNEL_STREAM_64)
            return run_stream<DT, 64, 1536, 16>(p, n, emb, fe, q, q_scale, b, row_bytes, k, fq, ps, pi, s);
    if (k <= 16)
        return run_stream<DT, 32, 3072, 16>(p, n, emb, fe, q, q_scale, b, row_bytes, k, fq, ps, pi, s);
    return run_stream<DT, 32, 3072, 64>(p, n, emb, fe, q, q_scale, b, row_bytes, k, fq, ps, pi, s);
}

}  // namespace

hipError_t launch_stream(const MatchPlan& p, int dt, int64_t n, int32_t d, const void* emb,
                         const float* fe, const void* q, const float* q_scale, int32_t b, int32_t k,
                         float* fq, float* ps, int* pi, hipStream_t s)
{
    const int64_t row_bytes = (int64_t)d * elem_bytes(dt);
    switch (dt) {
    case APC_F32: return run_stream_dt<APC_F32>(p, n, emb, fe, q, q_scale, b, row_bytes, k, fq, ps, pi, s);
    case APC_F16: return run_stream_dt<APC_F16>(p, n, emb, fe, q, q_scale, b, row_bytes, k, fq, ps, pi, s);
    case APC_BF16: return run_stream_dt<APC_BF16>(p, n, emb, fe, q, q_scale, b, row_bytes, k, fq, ps, pi, s);
    default: return run_stream_dt<APC_E4M3>(p, n, emb, fe, q, q_scale, b, row_bytes, k, fq, ps, pi, s);
    }
}

}  // namespace apc
