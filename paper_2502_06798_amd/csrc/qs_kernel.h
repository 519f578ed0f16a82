// Query-stationary similarity + exact top-k for 16-bit and e4m3 rows.
//
// Grid: splits x query tiles.  A workgroup of four wavefronts (one per SIMD)
// owns a tile of 4 x MQ x 32 queries and a contiguous range of cache entries
// (its split).  Each wavefront keeps its MQ x 32 query rows in VGPRs for its
// whole life, as the B operands of 32x32 MFMAs (lane l supplies query row
// l % 32; half h = l / 32 supplies bytes [64h, 64h + 64) of every 128-byte
// chunk of d), loaded from a copy that the query preparation writes in the
// order of these loads.  Cache rows stream through an LDS ring in stages of EB x 32
// rows x 256 bytes, loaded straight from global memory into LDS (no VGPRs held
// by loads in flight); a 16-byte unit of a row sits at unit ^ (row % 16), so
// the A-operand reads (lane = row) are free of bank conflicts.  One barrier
// per stage makes the stage visible to the four wavefronts, which all use it.
// The EB 32-row blocks of a stage give each wavefront EB x MQ independent
// accumulation chains (EB = 4 with one query block, 2 with two); every score
// is the sum over all of d in float32, in the same order whatever the split
// or tile.
//
// Top-k, per wavefront (its queries are its own, so no cross-wave sync).
// The two lanes of a query see disjoint entries; each keeps its own list of
// the best pairs it has seen, as order-preserving 64-bit keys: in registers,
// sorted, holding the KR best (LDS lists, unsorted, for 1024-byte rows with
// two query blocks).  After each group of EB x 32 entries:
//  * a lane's best score in the group is computed exactly (largest product
//    times entry factor, times f_q, clamped: both steps are monotone), and
//    only if it reaches the filter threshold does the lane look further;
//  * the filter threshold is the largest known lower bound on the query's
//    k-th best score: the pair's bound (either lane's k-th, and in a split's
//    first groups the smaller of one lane's ceil(k/2)-th and the other's
//    floor(k/2)-th) and a per-query bound shared by all workgroups through
//    atomic max (a published value has k entries scoring at least that
//    much; ties with it are kept).  The shared bound is read as late as the
//    LDS ring allows (with the next group's first stage), so that it
//    includes what other workgroups found meanwhile;
//  * each pair's exact score is tested against it (one multiply and one
//    compare), and the pairs that reach it go into the lane's list, one per
//    pass.
// At the end each lane's list is merged with its partner's, and the k best
// are written as the split's partial list; k_topk_merge merges the splits.
#pragma once

#include <type_traits>

#include "topk_wg.h"

namespace apc {
namespace {

typedef __attribute__((address_space(3))) void lds_void;

constexpr int Q2_NW = 4;                   // wavefronts per workgroup
constexpr int Q2_NT = Q2_NW * 64;
constexpr int Q2_SB = 256;                 // bytes of each row per stage
constexpr int Q2_FR = 8;                   // ring of per-group side data
constexpr int Q2_KMAX = 32;                // largest k
constexpr int Q2_LDS = 160 * 1024;         // LDS of a CU
// s_waitcnt immediate: at most n vector-memory operations outstanding
constexpr int Q2_PAIR_GROUPS = 8;          // groups of a split that bound the pair from both lists
constexpr int q2_vmcnt(int n) { return (n & 15) | (((n >> 4) & 3) << 14) | (7 << 4) | (15 << 8); }

// 16 bytes per lane from global memory straight into LDS: lane l's bytes land
// at lds + 16 l.  An asm statement, so that the compiler does not make every
// later LDS read wait for all loads in flight; the kernel counts them itself.
__device__ inline void q2_dma16(const void* g, uint32_t lds)
{
    asm volatile("s_nop 0\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(g), "{m0}"(lds) : "memory");
}

// the same, coherent across the device (values other workgroups update with
// device-scope atomics; plain loads could hit a stale line in this XCD's L2)
__device__ inline void q2_dma16_fresh(const void* g, uint32_t lds)
{
    asm volatile("s_nop 0\n\tglobal_load_lds_dwordx4 %0, off sc1" ::"v"(g), "{m0}"(lds) : "memory");
}

// order-preserving int image of a float (for atomicMax on scores)
__device__ inline int q2_key(float f)
{
    const int i = __float_as_int(f);
    return i >= 0 ? i : i ^ 0x7fffffff;
}
__device__ inline float q2_unkey(int k) { return __int_as_float(k >= 0 ? k : k ^ 0x7fffffff); }

// fire-and-forget atomic max (no return value, nothing to wait for)
__device__ inline void q2_atomic_max(int* p, int v)
{
    asm volatile("global_atomic_smax %0, %1, off" ::"v"(p), "v"(v) : "memory");
}

// an empty asm statement that reads x from VGPRs (x is 16 or 32 bytes)
template <class T>
__device__ inline void q2_use(const T& x)
{
    typedef int v4 __attribute__((ext_vector_type(4)));
    typedef int v8 __attribute__((ext_vector_type(8)));
    if constexpr (sizeof(T) == 16) asm volatile("" ::"v"(__builtin_bit_cast(v4, x)));
    else asm volatile("" ::"v"(__builtin_bit_cast(v8, x)));
}

template <int DT> struct Q2Op { typedef uint4 Step; static constexpr int UPS = 1; };
template <> struct Q2Op<APC_E4M3> { typedef i32x8 Step; static constexpr int UPS = 2; };

// f(integral_constant<int, 0>) ... f(integral_constant<int, N - 1>)
template <int N, int I = 0, class Fn>
__device__ inline __attribute__((always_inline)) void static_for(Fn&& f)
{
    if constexpr (I < N) {
        f(std::integral_constant<int, I>{});
        static_for<N, I + 1>(f);
    }
}

struct Q2Pair {
    float s;
    int i;
};

template <int DT, int RB, int MQ, int KR, int EB>
struct Q2Cfg {
    typedef typename Q2Op<DT>::Step Step;
    static constexpr int UPS = Q2Op<DT>::UPS;         // 16-byte units per MFMA step
    static constexpr int SPG = RB / Q2_SB;            // stages per group
    static constexpr int SST = Q2_SB / 32 / UPS;      // MFMA steps per stage (per block)
    static constexpr int QST = RB / 32 / UPS;         // steps of a query row held by a lane
    static constexpr int BQW = MQ * 32;               // queries per wavefront
    static constexpr int BQ = Q2_NW * BQW;            // queries per workgroup
    static constexpr int GR = EB * 32;                // rows per stage and per group (EB blocks of 32)
    static constexpr int STAGE = GR * Q2_SB;          // bytes of a stage
    static constexpr int LPW = STAGE / 1024 / Q2_NW;  // row loads per wavefront per stage
    static constexpr bool LREG = MQ == 1 || RB < 1024; // lists in registers (else LDS)
    static constexpr bool LLDS = !LREG;               // lists in LDS
    static constexpr int LIST_BYTES = LLDS ? Q2_NW * MQ * KR * 64 * 8 : 0;
    static constexpr int SIDE_BYTES = Q2_FR * GR * 4 + Q2_FR * Q2_NW * BQW * 4;
    static constexpr int NS = (Q2_LDS - LIST_BYTES - SIDE_BYTES) / STAGE;   // stages in the LDS ring
    static_assert(NS >= 4, "LDS ring too small");
    static_assert(EB == 2 || EB == 4, "two or four blocks per group");
    static_assert(RB % Q2_SB == 0 && SPG >= 2, "rows must be at least two whole stages");
    static_assert(STAGE % (1024 * Q2_NW) == 0, "stage loads split evenly over the wavefronts");
    // stages s = t + d, d in [d0, d1], with s % SPG == r, for t % SPG == j
    static constexpr int count_at(int j, int d0, int d1, int r)
    {
        int c = 0;
        for (int d = d0; d <= d1; ++d) c += ((j + d) % SPG + SPG) % SPG == r;
        return c;
    }
    // Loads of a group's first stage s: the previous group's global bounds (for
    // its epilogue, read as late as the ring allows), then the rows, then the
    // group's entry factors.  Vector-memory operations a wavefront issues after
    // stage t's row loads and before it waits for stage t (j = t % SPG): the
    // rows of stages t + 1 .. t + NS - 2, entry factors for first stages s in
    // [t, t + NS - 2], bounds for first stages s in [t + 1, t + NS - 2].
    static constexpr int after(int j)
    {
        return (NS - 2) * LPW + count_at(j, 0, NS - 2, 0) + count_at(j, 1, NS - 2, 0);
    }
    // at a group's epilogue, the operations issued after its global bounds: the
    // loads of the next NS - 1 stages (starting with the next group's first)
    static constexpr int after_bounds()
    {
        return (NS - 1) * LPW + count_at(0, 0, NS - 2, 0) + count_at(0, 1, NS - 2, 0);
    }
    template <int J>
    __device__ static void wait_stage() { __builtin_amdgcn_s_waitcnt(q2_vmcnt(after(J))); }
    struct Smem {
        uint8_t e[NS * STAGE];
        float fe[Q2_FR][GR];                    // entry factors of a group
        int gthr[Q2_FR][Q2_NW][BQW];            // global bounds (keys) seen at a group start
        uint64_t lst[LLDS ? Q2_NW : 1][MQ][LLDS ? KR : 1][64];   // per-lane lists of keys (LDS form), slot-major
    };
};

// c += a b; first: c = a b (the accumulator input is the constant 0, so the
// accumulators need no clearing between groups; first is a constant once the
// step loops are unrolled)
template <int DT>
__device__ inline void q2_mma(f32x16& c, const typename Q2Op<DT>::Step a, const typename Q2Op<DT>::Step b, bool first)
{
    const f32x16 cin = first ? f32x16{} : c;
    if constexpr (DT == APC_F16)
        c = __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(f16x8, a), __builtin_bit_cast(f16x8, b), cin, 0, 0, 0);
    else if constexpr (DT == APC_BF16)
        c = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), cin, 0, 0, 0);
    else
        c = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, b, cin, 0, 0, 0, 0, 0, 0);
}

// A (score, entry) pair as one 64-bit key ordered like (score desc, entry
// asc): the high word is the score's bits mapped to an order-preserving
// unsigned integer, the low word the complement of the entry index.  Key 0
// marks an empty slot (below every pair).
__device__ inline uint64_t q2_pack(float s, int e)
{
    const uint32_t u = __float_as_uint(s);
    const uint32_t o = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
    return ((uint64_t)o << 32) | (uint32_t)~(uint32_t)e;
}
__device__ inline float q2_key_score(uint64_t key)
{
    if (key == 0) return neg_inf();
    const uint32_t o = (uint32_t)(key >> 32);
    return __uint_as_float((o & 0x80000000u) ? (o & 0x7fffffffu) : ~o);
}
__device__ inline int q2_key_entry(uint64_t key) { return key == 0 ? IDX_NONE : (int)~(uint32_t)key; }

// smallest key of a lane's list (slots past k hold ~0 and are never the smallest):
// all KR slots are read at once, then a tree of comparisons
template <int KR>
__device__ inline void q2_worst(const uint64_t* col, uint64_t& wkey, int& wp)
{
    uint64_t x[KR];
    int xp[KR];
#pragma unroll
    for (int p = 0; p < KR; ++p) {
        x[p] = col[p * 64];
        xp[p] = p;
    }
#pragma unroll
    for (int w = 1; w < KR; w *= 2)
#pragma unroll
        for (int p = 0; p + w < KR; p += 2 * w) {
            const bool tk = x[p + w] < x[p];
            x[p] = tk ? x[p + w] : x[p];
            xp[p] = tk ? xp[p + w] : xp[p];
        }
    wkey = x[0];
    wp = xp[0];
}

// register form, kept sorted by key descending: insert key (0 inserts
// nothing), dropping the smallest.  Every slot compares once; a slot takes the
// one before it when the key goes above that one, the key when it goes above
// only this one.  Slots are written from the last up, so each new value can
// take the old one's register.
template <int KR>
__device__ inline void q2_insert_sorted(uint64_t (&lk)[KR], uint64_t key)
{
    bool above[KR];
#pragma unroll
    for (int p = 0; p < KR; ++p) above[p] = key > lk[p];
#pragma unroll
    for (int p = KR - 1; p > 0; --p) lk[p] = above[p - 1] ? lk[p - 1] : (above[p] ? key : lk[p]);
    lk[0] = above[0] ? key : lk[0];
}

// 2 m + c in one instruction: the compare result c enters as the carry
__device__ inline uint32_t q2_shift_in(uint32_t m, bool c)
{
    uint32_t r;
    uint64_t carry_out;
    asm("v_addc_co_u32_e64 %0, %1, %2, %2, %3" : "=v"(r), "=s"(carry_out) : "v"(m), "s"(__builtin_amdgcn_ballot_w64(c)));
    return r;
}

// (m & x) | (~m & y) for a mask m of all zeros or all ones (one v_bfi_b32).
// The mask goes through an empty asm so that the optimizer cannot see it is
// a select and fold a tree of them into one dynamically indexed read, which
// would go through scratch memory.
__device__ inline uint32_t q2_opaque(uint32_t m)
{
    asm("" : "+v"(m));
    return m;
}
__device__ inline float q2_bsel(uint32_t m, float x, float y)
{
    return __uint_as_float((__float_as_uint(x) & m) | (__float_as_uint(y) & ~m));
}

// slot i (the same for the whole wavefront, below KR) of a register list,
// through a tree of bit selects
template <int KR>
__device__ inline uint64_t q2_slot(const uint64_t (&lk)[KR], int i)
{
    uint32_t lo[KR], hi[KR];
#pragma unroll
    for (int p = 0; p < KR; ++p) {
        lo[p] = (uint32_t)lk[p];
        hi[p] = (uint32_t)(lk[p] >> 32);
    }
#pragma unroll
    for (int w = 1; w < KR; w *= 2) {
        const uint32_t m = q2_opaque(0u - (uint32_t)((i / w) & 1));
#pragma unroll
        for (int p = 0; p + w < KR; p += 2 * w) {
            lo[p] = __float_as_uint(q2_bsel(m, __uint_as_float(lo[p + w]), __uint_as_float(lo[p])));
            hi[p] = __float_as_uint(q2_bsel(m, __uint_as_float(hi[p + w]), __uint_as_float(hi[p])));
        }
    }
    return ((uint64_t)hi[0] << 32) | lo[0];
}

// the 16 EB values v[eb][r] of a lane, element b = 16 eb + r, chosen by the
// bits of b through a tree of bit selects (ordinary selects would be folded
// into one dynamically indexed read, which goes through scratch memory)
template <int EB>
__device__ inline float q2_pick(const f32x16 (&v)[EB], int b)
{
    const uint32_t m0 = q2_opaque(0u - (uint32_t)(b & 1)), m1 = q2_opaque(0u - (uint32_t)((b >> 1) & 1));
    const uint32_t m2 = q2_opaque(0u - (uint32_t)((b >> 2) & 1)), m3 = q2_opaque(0u - (uint32_t)((b >> 3) & 1));
    const uint32_t m4 = q2_opaque(0u - (uint32_t)((b >> 4) & 1));
    float l16[16], l8[8], l4[4];
#pragma unroll
    for (int i = 0; i < 16; ++i) {
        if constexpr (EB == 2) {
            l16[i] = q2_bsel(m4, v[1][i], v[0][i]);
        } else {
            const uint32_t m5 = q2_opaque(0u - (uint32_t)((b >> 5) & 1));
            l16[i] = q2_bsel(m5, q2_bsel(m4, v[3][i], v[2][i]), q2_bsel(m4, v[1][i], v[0][i]));
        }
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) l8[i] = q2_bsel(m0, l16[2 * i + 1], l16[2 * i]);
#pragma unroll
    for (int i = 0; i < 4; ++i) l4[i] = q2_bsel(m1, l8[2 * i + 1], l8[2 * i]);
    const float l2a = q2_bsel(m2, l4[1], l4[0]), l2b = q2_bsel(m2, l4[3], l4[2]);
    return q2_bsel(m3, l2b, l2a);
}

// grid: workgroup id -> (split, query tile).  With a grid that is a multiple
// of 8, consecutive linear indices go to the same XCD (workgroups are dealt
// round-robin over the 8 XCDs), so the query tiles of a split run side by
// side on one XCD and share its L2.
template <int DT, int RB, int MQ, int KR, int EB>
__global__ __launch_bounds__(Q2_NT) void k_qs(
    const uint8_t* __restrict__ emb, const float* __restrict__ fe, int64_t n,
    const uint8_t* __restrict__ qry, const float* __restrict__ fq_ws, int* __restrict__ gthr, int32_t b,
    int32_t k, int splits, int qtiles, int64_t b_pad, float* __restrict__ part_s, int* __restrict__ part_i)
{
    typedef Q2Cfg<DT, RB, MQ, KR, EB> C;
    typedef typename C::Step Step;
    constexpr int NS = C::NS, SPG = C::SPG, SST = C::SST, UPS = C::UPS, BQW = C::BQW;
    constexpr int GR = C::GR, STAGE = C::STAGE, LPW = C::LPW;
    typedef typename std::conditional<EB == 4, uint64_t, uint32_t>::type Mask;   // one bit per value of a lane
    __shared__ typename C::Smem sm;
    const int tid = threadIdx.x, lane = tid & 63, h = lane >> 5, r32 = lane & 31;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);

    const int grid = (int)gridDim.x, work = splits * qtiles;
    const int lin = (grid & 7) == 0 ? (int)(blockIdx.x & 7) * (grid >> 3) + (int)(blockIdx.x >> 3) : (int)blockIdx.x;
    if (lin >= work) return;                                       // whole workgroup: uniform
    const int split = lin / qtiles, qtile = lin % qtiles;
    const int64_t q0w = (int64_t)qtile * C::BQ + wave * BQW;      // this wavefront's first query
    const bool live = q0w < b;                                     // uniform per wavefront

    const int64_t ngr = (n + GR - 1) / GR;                         // groups of the cache
    const int64_t g_begin = ngr * split / splits;
    const int ng = (int)(ngr * (split + 1) / splits - g_begin);   // groups of this split (>= 1)
    const int T = ng * SPG;                                        // stages of this split

    // ---- stage loads: wavefront w fills rows [w GR/4, (w + 1) GR/4) of a stage ----
    const uint32_t lds_e = (uint32_t)(size_t)(lds_void*)sm.e;
    const uint32_t lds_fe = (uint32_t)(size_t)(lds_void*)&sm.fe[0][0];
    const uint32_t lds_gt = (uint32_t)(size_t)(lds_void*)&sm.gthr[0][0][0];
    int lrow[LPW], loff[LPW];
#pragma unroll
    for (int i = 0; i < LPW; ++i) {
        lrow[i] = wave * (GR / Q2_NW) + i * 4 + (lane >> 4);
        loff[i] = ((lane & 15) ^ (lrow[i] & 15)) * 16;             // logical unit stored at unit lane % 16
    }
    // row pointers of the group being issued (groups are issued in order); a
    // stage j of the group adds j * 256 to them (not through the load's offset
    // field: for loads into LDS that offset moves the LDS address too)
    const uint8_t* rowp[LPW];
    // Part p of NP (SST - LA + 1 or 1) issues the bounds (p = 0),
    // the row loads i with i % NP == p, then the entry factors (p = NP - 1),
    // in that order; a negative part issues everything.  The stage loop issues part p at its
    // step p, all before its wait for the next stage, so the order of the
    // loads, and with it every wait count, is that of issuing them at once.
    constexpr int LA = SST < 3 ? SST : 2;
    // (spread only for 16-bit rows with one query block per wavefront: e4m3
    // rows run out of registers, and with two blocks, four MFMAs per step,
    // spreading was slower)
    constexpr int NP = UPS == 1 && MQ == 1 ? SST - LA + 1 : 1;
    auto issue = [&](int gi, auto jc, int part) __attribute__((always_inline)) {                  // stage j of group gi
        constexpr int j = decltype(jc)::value;
        const bool all = part < 0;
        if constexpr (j == 0) {
            if (gi >= 1 && (all || part == 0)) {
                // the previous group's global bounds, for its epilogue: this
                // wavefront's queries, one load, lanes beyond the data idle
                const int gl = lane < BQW / 4 ? lane : 0;
                if (lane < BQW / 4)
                    q2_dma16_fresh(gthr + q0w + gl * 4,
                                   lds_gt + (uint32_t)((((gi - 1) % Q2_FR) * Q2_NW + wave) * BQW * 4));
            }
            if (gi * SPG >= T) return;                             // past the last stage: bounds only
        }
        const int64_t e0 = (g_begin + gi) * GR;
        if constexpr (j == 0) {
            if (all || part == 0) {
                const int64_t last = n - 1 - e0;                   // last valid row of the group
#pragma unroll
                for (int i = 0; i < LPW; ++i) {
                    const int64_t row = lrow[i] < last ? lrow[i] : last;
                    rowp[i] = emb + (e0 + row) * RB + loff[i];
                }
            }
        }
        const int t = gi * SPG + j;
        const uint32_t sbase = lds_e + (uint32_t)(t % NS) * STAGE;
#pragma unroll
        for (int i = 0; i < LPW; ++i)
            if (all || i % NP == part)
                q2_dma16(rowp[i] + j * Q2_SB, __builtin_amdgcn_readfirstlane(
                                                  sbase + (uint32_t)(wave * (GR / Q2_NW) + i * 4) * Q2_SB));
        if constexpr (j == 0) {
            // the group's GR entry factors (zero-padded to whole groups): one load,
            // lanes beyond the data idle
            const int fl = lane < GR / 4 ? lane : 0;
            if ((all || part == NP - 1) && lane < GR / 4)
                q2_dma16(fe + e0 + fl * 4, lds_fe + (uint32_t)(gi % Q2_FR) * (GR * 4));
        }
    };
    // stage s = t0 + d of the schedule, with t0 = gi0 * SPG + j0 (j0, d compile-time)
    auto issue_ahead = [&](int gi0, auto j0c, auto dc, int part) __attribute__((always_inline)) {
        constexpr int js = (decltype(j0c)::value + decltype(dc)::value) % SPG;
        constexpr int dg = (decltype(j0c)::value + decltype(dc)::value) / SPG;
        issue(gi0 + dg, std::integral_constant<int, js>{}, part);
    };
    static_for<NS - 1>([&](auto sc) __attribute__((always_inline)) {
        if (decltype(sc)::value <= T) issue_ahead(0, std::integral_constant<int, 0>{}, sc, -1);
    });

    // ---- queries into VGPRs, factors, empty lists ----
    // The queries come in load order (written by the query preparation):
    // block mq of this wavefront, step s, is 64 consecutive Steps, one per lane.
    Step qv[C::QST][MQ];
    float fq[MQ];
#pragma unroll
    for (int mq = 0; mq < MQ; ++mq) {
        const int64_t qg = q0w + mq * 32 + r32;
        const uint8_t* qblk = qry + ((((int64_t)qtile * Q2_NW + wave) * MQ + mq) * C::QST * 64 + lane) * sizeof(Step);
#pragma unroll
        for (int s = 0; s < C::QST; ++s) qv[s][mq] = *reinterpret_cast<const Step*>(qblk + (int64_t)s * 64 * sizeof(Step));
        fq[mq] = fq_ws[qg];                          // NaN for rows that cannot be matched
    }
    // The compiler waits for these loads here: every value is used by an empty
    // asm statement, so the loads cannot sink into the main loop, where the
    // wait for them (counted without the LDS loads) would drain those as well.
#pragma unroll
    for (int s2 = 0; s2 < C::QST; ++s2)
#pragma unroll
        for (int mq = 0; mq < MQ; ++mq) q2_use(qv[s2][mq]);
#pragma unroll
    for (int mq = 0; mq < MQ; ++mq) asm volatile("" ::"v"(fq[mq]));
    // per-lane lists.  Registers: the KR best keys, sorted descending (key 0:
    // empty).  LDS: slots below k start empty, slots from k on hold ~0 so that
    // they are never the worst.
    constexpr bool LREG = C::LREG;
    uint64_t* lcol[MQ];
    uint64_t lk[LREG ? MQ : 1][KR];
#pragma unroll
    for (int mq = 0; mq < MQ; ++mq) {
        if constexpr (LREG) {
#pragma unroll
            for (int p = 0; p < KR; ++p) lk[mq][p] = 0ull;
        } else {
            lcol[mq] = &sm.lst[wave][mq][0][lane];
#pragma unroll
            for (int p = 0; p < KR; ++p) lcol[mq][p * 64] = p < k ? 0ull : ~0ull;
        }
    }
    uint64_t wkey[MQ];   // the lane's k-th key (0 while it has fewer than k)
    int wp[MQ];          // its slot (lists in LDS)
    float ps[MQ];        // a lower bound on the query's k-th best from the pair's lists (-inf until known)
#pragma unroll
    for (int mq = 0; mq < MQ; ++mq) {
        wkey[mq] = 0;
        wp[mq] = 0;
        ps[mq] = neg_inf();
    }

    f32x16 acc[MQ][EB];      // written whole by each group's first MFMA step

    // the stages of logical group gi (every wavefront, for the loads and
    // barriers).  The A fragments of step ss (all EB blocks) are read LA steps
    // ahead of the MFMAs that use them; a scheduling barrier after each step
    // keeps the compiler from regrouping the MFMAs by accumulator, which would
    // wait out every read's latency and every MFMA's.  Within a group, the wait
    // and barrier for the next stage come LA steps before the end of a stage,
    // and the next stage's first LA reads go out while its last MFMAs run, so
    // the matrix unit does not idle across the barrier.  Nothing is issued
    // between the two points, so the wait counts are those of the next stage;
    // the barrier comes after all of this stage's reads (it waits for them),
    // so the next stage may refill this stage's slot.
    auto run_group = [&](int gi) __attribute__((always_inline)) {
        Step an[LA][EB];                                           // the next stage's first fragments
        static_for<SPG>([&](auto jc) __attribute__((always_inline)) {
            constexpr int j = decltype(jc)::value;
            constexpr bool early = j > 0;                          // wait, barrier, first reads done already
            constexpr bool ahead = j + 1 < SPG;                    // do them for the next stage here
            const int t = gi * SPG + j;
            if constexpr (!early) {
                if (t + NS - 2 < T) C::template wait_stage<j>();
                else __builtin_amdgcn_s_waitcnt(q2_vmcnt(0));
                __syncthreads();
            }
            auto wait_next = [&]() __attribute__((always_inline)) {
                if constexpr (ahead) {
                    if (t + 1 + NS - 2 < T) C::template wait_stage<(ahead ? j + 1 : 0)>();
                    else __builtin_amdgcn_s_waitcnt(q2_vmcnt(0));
                    __syncthreads();
                }
            };
            const uint8_t* sb = sm.e + (t % NS) * STAGE + r32 * Q2_SB;
            const uint8_t* sbn = sm.e + ((t + 1) % NS) * STAGE + r32 * Q2_SB;
            Step a[SST][EB];
            auto rd = [&](const uint8_t* base, int ss, Step (&dst)[EB]) __attribute__((always_inline)) {
                const int cl = ss / (4 / UPS), sp = (ss % (4 / UPS)) * UPS;
                const int lu = cl * 8 + h * 4 + sp;                      // logical 16-byte unit
#pragma unroll
                for (int eb = 0; eb < EB; ++eb) {
                    const uint8_t* rp = base + eb * 32 * Q2_SB;
                    if constexpr (UPS == 1) {
                        dst[eb] = *reinterpret_cast<const uint4*>(rp + ((lu ^ (r32 & 15)) * 16));
                    } else {
                        const uint4 x0 = *reinterpret_cast<const uint4*>(rp + ((lu ^ (r32 & 15)) * 16));
                        const uint4 x1 = *reinterpret_cast<const uint4*>(rp + (((lu + 1) ^ (r32 & 15)) * 16));
                        dst[eb] = Step{(int)x0.x, (int)x0.y, (int)x0.z, (int)x0.w,
                                       (int)x1.x, (int)x1.y, (int)x1.z, (int)x1.w};
                    }
                }
            };
            // the first reads go out before the stage loads are issued
            if (live) {
#pragma unroll
                for (int ss = 0; ss < LA; ++ss) {
                    if constexpr (early) {
#pragma unroll
                        for (int eb = 0; eb < EB; ++eb) a[ss][eb] = an[ss][eb];
                    } else {
                        rd(sb, ss, a[ss]);
                    }
                }
            }
            const bool issue_now = t + NS - 1 <= T;                // into the slot stage t - 1 used
            if (issue_now && (NP == 1 || !live))
                issue_ahead(gi, std::integral_constant<int, j>{}, std::integral_constant<int, NS - 1>{}, -1);
            if (!live) {
                wait_next();
                return;
            }

#pragma unroll
            for (int ss = 0; ss < SST; ++ss) {
                if (NP > 1 && ss < NP && issue_now)
                    issue_ahead(gi, std::integral_constant<int, j>{}, std::integral_constant<int, NS - 1>{}, ss);
                if (ss + LA < SST) rd(sb, ss + LA, a[ss + LA]);
                if constexpr (ahead) {
                    if (ss == SST - LA) wait_next();
                    if (ss >= SST - LA) rd(sbn, ss - (SST - LA), an[ss - (SST - LA)]);
                }
#pragma unroll
                for (int eb = 0; eb < EB; ++eb)
#pragma unroll
                    for (int mq = 0; mq < MQ; ++mq) q2_mma<DT>(acc[mq][eb], a[ss][eb], qv[j * SST + ss][mq], j == 0 && ss == 0);
                __builtin_amdgcn_sched_barrier(0);
            }
        });
    };
    for (int gi = 0; gi < ng; ++gi) {
        run_group(gi);
        if (!live) continue;
        // the group's global bounds (loaded with the next group's first stage)
        if ((gi + 1) * SPG + NS - 2 < T) __builtin_amdgcn_s_waitcnt(q2_vmcnt(C::after_bounds()));
        else __builtin_amdgcn_s_waitcnt(q2_vmcnt(0));

        // ---- epilogue of the group ----
        // lane (h, c) holds for query c the rows 8 g + 4 h + i (g, i < 4) of each
        // block; quad p = 4 eb + g groups its four rows i
        const int64_t e0 = (g_begin + gi) * GR;
        const bool whole = e0 + GR <= n;
        const int64_t lim64 = n - e0 - 4 * h;                  // rows 8g + i (+ 32 eb) below this are < n
        const float* fr = sm.fe[gi % Q2_FR];             // the group's entry factors
        // The filter threshold F is the largest valid lower bound on the query's
        // k-th best score: the lane's own k-th, its partner lane's, the global one.
        // The lane's best score in the group is computed exactly: its largest
        // product times entry factor, then times f_q and clamped (both monotone).
        // The products times entry factor stay in acc for the exact test below.
        // Rows past n read the zero padding of the factors, which at most lets
        // the group through to that test.
        float m[MQ];
#pragma unroll
        for (int mq = 0; mq < MQ; ++mq) m[mq] = neg_inf();
#pragma unroll
        for (int eb = 0; eb < EB; ++eb) {
            float fv[16];
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                const float4 f4 = *reinterpret_cast<const float4*>(fr + eb * 32 + 8 * g + 4 * h);
                fv[4 * g] = f4.x;
                fv[4 * g + 1] = f4.y;
                fv[4 * g + 2] = f4.z;
                fv[4 * g + 3] = f4.w;
            }
#pragma unroll
            for (int mq = 0; mq < MQ; ++mq)
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const float x = acc[mq][eb][r] * fv[r];
                    acc[mq][eb][r] = x;
                    m[mq] = __builtin_fmaxf(m[mq], x);
                }
        }
        if (gi == 0 && k <= 16) {
            // Seed for the first group (the lists are still empty): the 8 EB quads
            // of a lane pair are disjoint, so the k-th largest of the pair's quad
            // maxima has k pairs at or above it.  For k <= 4 EB it is found by
            // merging the two lanes' sorted maxima; above that, the smaller of one
            // lane's ceil(k/2)-th largest and the other's floor(k/2)-th serves.
            constexpr int NQ = 4 * EB;                             // quads per lane
#pragma unroll
            for (int mq = 0; mq < MQ; ++mq) {
                float qm[NQ];
#pragma unroll
                for (int eb = 0; eb < EB; ++eb)
#pragma unroll
                    for (int g = 0; g < 4; ++g) {
                        float x = neg_inf();
#pragma unroll
                        for (int i = 0; i < 4; ++i)
                            if (whole || 32 * eb + 8 * g + i < lim64)
                                x = __builtin_fmaxf(x, acc[mq][eb][4 * g + i]);
                        qm[4 * eb + g] = x;
                    }
                // sort descending (bitonic)
#pragma unroll
                for (int size = 2; size <= NQ; size *= 2)
#pragma unroll
                    for (int stride = size / 2; stride > 0; stride /= 2)
#pragma unroll
                        for (int i = 0; i < NQ; ++i) {
                            const int j = i ^ stride;
                            if (j > i) {
                                const bool desc = (i & size) == 0;
                                const float a0 = qm[i], a1 = qm[j];
                                const bool sw = desc ? a0 < a1 : a0 > a1;
                                qm[i] = sw ? a1 : a0;
                                qm[j] = sw ? a0 : a1;
                            }
                        }
                float seed;
                if (k <= NQ) {                                     // uniform
                    // own maxima (descending) against the partner's reversed form a
                    // bitonic sequence whose larger elements are the NQ largest of
                    // both; half-cleaners sort them
                    float u[NQ];
#pragma unroll
                    for (int p = 0; p < NQ; ++p) u[p] = __builtin_fmaxf(qm[p], __shfl_xor(qm[NQ - 1 - p], 32, 64));
#pragma unroll
                    for (int stride = NQ / 2; stride > 0; stride /= 2)
#pragma unroll
                        for (int i = 0; i < NQ; ++i)
                            if ((i & stride) == 0) {
                                const float hi = __builtin_fmaxf(u[i], u[i + stride]);
                                const float lo = __builtin_fminf(u[i], u[i + stride]);
                                u[i] = hi;
                                u[i + stride] = lo;
                            }
                    seed = u[0];
#pragma unroll
                    for (int p = 1; p < NQ; ++p) seed = p == k - 1 ? u[p] : seed;
                } else {
                    const int m1 = (k + 1) / 2, m2 = k - m1;      // 1 <= m1, m2 <= 8
                    float a1 = qm[0], a2 = qm[0];
#pragma unroll
                    for (int p = 1; p < NQ; ++p) {
                        a1 = p == m1 - 1 ? qm[p] : a1;
                        a2 = p == m2 - 1 ? qm[p] : a2;
                    }
                    const float b1 = __shfl_xor(a1, 32, 64), b2 = __shfl_xor(a2, 32, 64);
                    seed = __builtin_fmaxf(__builtin_fminf(a1, b2), __builtin_fminf(b1, a2));
                }
                // as a score (NaN f_q leaves the seed at -inf through the comparison below)
                const float ss = clamp1(seed * fq[mq]);
                if (ss > ps[mq]) ps[mq] = ss;
            }
        }
        float G[MQ], F[MQ];
        bool pass[MQ];
        bool any_pass = false;
#pragma unroll
        for (int mq = 0; mq < MQ; ++mq) {
            G[mq] = q2_unkey(sm.gthr[gi % Q2_FR][wave][mq * 32 + r32]);
            F[mq] = __builtin_fmaxf(__builtin_fmaxf(q2_key_score(wkey[mq]), ps[mq]), G[mq]);
            pass[mq] = fq[mq] == fq[mq] && clamp1(m[mq] * fq[mq]) >= F[mq];   // NaN f_q: row not matched
            any_pass |= pass[mq];
        }
        if (__builtin_amdgcn_ballot_w64(any_pass)) {
            // rows below n, bit 16 eb + r for row 32 eb + 8 (r / 4) + 4 h + r % 4
            Mask valid = ~(Mask)0;
            if (!whole) {
                valid = 0;
#pragma unroll
                for (int eb = 0; eb < EB; ++eb)
#pragma unroll
                    for (int r = 0; r < 16; ++r)
                        if (32 * eb + 8 * (r >> 2) + (r & 3) < lim64) valid |= (Mask)1 << (16 * eb + r);
            }
#pragma unroll
            for (int mq = 0; mq < MQ; ++mq) {
                // the pairs whose exact score reaches F.  Scores are at least -1, so
                // with F <= -1 every row passes; otherwise clamp1(y) >= F exactly when
                // y >= F (F <= 1, and a NaN product fails both).  The bits are shifted
                // in from the highest row of each 32-bit word down.
                Mask mask = 0;
                if (pass[mq]) {
                    if (F[mq] <= -1.f) {
                        mask = valid;
                    } else {
                        uint32_t w[(EB * 16 + 31) / 32];
#pragma unroll
                        for (int wi = 0; wi < (EB * 16 + 31) / 32; ++wi) {
                            uint32_t b = 0;
#pragma unroll
                            for (int j = 31; j >= 0; --j) {
                                const int el = 32 * wi + j;
                                b = q2_shift_in(b, acc[mq][el >> 4][el & 15] * fq[mq] >= F[mq]);
                            }
                            w[wi] = b;
                        }
                        if constexpr (EB == 4) mask = ((Mask)w[1] << 32 | w[0]) & valid;
                        else mask = w[0] & valid;
                    }
                }
                // every lane inserts into its own list, one pair per pass
                while (__builtin_amdgcn_ballot_w64(mask != 0)) {
                    const bool act = mask != 0;
                    const int bsel = act ? (EB == 4 ? __builtin_ctzll((uint64_t)mask) : __builtin_ctz((uint32_t)mask)) : 0;
                    mask &= mask - 1;
                    const float sc = clamp1(q2_pick<EB>(acc[mq], bsel) * fq[mq]);
                    const int r = bsel & 15;
                    const int e = (int)(e0 + 32 * (bsel >> 4) + 8 * (r >> 2) + 4 * h + (r & 3));
                    const uint64_t key = q2_pack(sc, e);
                    if constexpr (LREG) {
                        q2_insert_sorted<KR>(lk[mq], act ? key : 0ull);
                    } else if (act && key > wkey[mq]) {
                        lcol[mq][wp[mq] * 64] = key;
                        q2_worst<KR>(lcol[mq], wkey[mq], wp[mq]);
                    }
                }
                if constexpr (LREG) wkey[mq] = q2_slot<KR>(lk[mq], k - 1);
            }
        }
        // The pair's bound for the next group, and the global bound.  Besides
        // either lane's k-th, with sorted lists: the smaller of one lane's m-th
        // and the other's (k - m)-th best (m = ceil(k / 2)) has k pairs at or
        // above it, which is far tighter while the lists are short (the first
        // Q2_PAIR_GROUPS groups of a split; later it rarely beats the k-th and
        // costs two slot selects per group).
#pragma unroll
        for (int mq = 0; mq < MQ; ++mq) {
            const float own = q2_key_score(wkey[mq]);
            float pair = __builtin_fmaxf(own, __shfl_xor(own, 32, 64));
            if constexpr (LREG) {
                if (k >= 2 && gi < Q2_PAIR_GROUPS) {               // uniform
                    const int m1 = (k + 1) / 2, m2 = k - m1;
                    const uint64_t a = q2_slot<KR>(lk[mq], m1 - 1), c = q2_slot<KR>(lk[mq], m2 - 1);
                    const uint64_t pa = ((uint64_t)(uint32_t)__shfl_xor((int)(a >> 32), 32, 64) << 32) |
                                        (uint32_t)__shfl_xor((int)(uint32_t)a, 32, 64);
                    const uint64_t pc = ((uint64_t)(uint32_t)__shfl_xor((int)(c >> 32), 32, 64) << 32) |
                                        (uint32_t)__shfl_xor((int)(uint32_t)c, 32, 64);
                    const uint64_t t1 = a < pc ? a : pc, t2 = pa < c ? pa : c;
                    pair = __builtin_fmaxf(pair, q2_key_score(t1 > t2 ? t1 : t2));
                }
            }
            ps[mq] = pair;
            if (h == 0 && pair > G[mq]) q2_atomic_max(gthr + q0w + mq * 32 + r32, q2_key(pair));
        }
    }

    if (!live) return;
    // ---- the split's partial list of each query: sort each lane's list,
    // merge it with the partner lane's, lane half 0 writes the k best ----
#pragma unroll
    for (int mq = 0; mq < MQ; ++mq) {
        // the list padded with empty slots to a power of two
        constexpr int KP = KR <= 16 ? 16 : 32;
        uint64_t x[KP];
#pragma unroll
        for (int p = 0; p < KP; ++p) {
            uint64_t v = 0ull;
            if (p < KR) {
                if constexpr (LREG) v = lk[mq][p];
                else v = lcol[mq][p * 64];
            }
            x[p] = v == ~0ull ? 0ull : v;
        }
        // bitonic sort, descending (register lists are sorted already)
#pragma unroll
        for (int size = 2; size <= (LREG ? 1 : KP); size *= 2)
#pragma unroll
            for (int stride = size / 2; stride > 0; stride /= 2)
#pragma unroll
                for (int i = 0; i < KP; ++i) {
                    const int j = i ^ stride;
                    if (j > i) {
                        const bool desc = (i & size) == 0;
                        const bool sw = desc ? x[i] < x[j] : x[i] > x[j];
                        const uint64_t a0 = x[i], a1 = x[j];
                        x[i] = sw ? a1 : a0;
                        x[j] = sw ? a0 : a1;
                    }
                }
        // the larger of own[p] and partner[KP - 1 - p] is a bitonic sequence
        // holding the KP largest of both lists; half-cleaners sort it
        uint64_t m[KP];
#pragma unroll
        for (int p = 0; p < KP; ++p) {
            const uint64_t o = x[KP - 1 - p];
            const uint32_t lo = __shfl_xor((uint32_t)o, 32, 64), hi = __shfl_xor((uint32_t)(o >> 32), 32, 64);
            const uint64_t y = ((uint64_t)hi << 32) | lo;            // partner's (KP - 1 - p)-th
            m[p] = x[p] > y ? x[p] : y;
        }
#pragma unroll
        for (int stride = KP / 2; stride > 0; stride /= 2)
#pragma unroll
            for (int i = 0; i < KP; ++i)
                if ((i & stride) == 0) {
                    const bool sw = m[i] < m[i + stride];
                    const uint64_t a0 = m[i], a1 = m[i + stride];
                    m[i] = sw ? a1 : a0;
                    m[i + stride] = sw ? a0 : a1;
                }
        const int64_t qg = q0w + mq * 32 + r32;
        if (h == 0 && qg < b_pad) {
            const int64_t o = (qg * splits + split) * k;
#pragma unroll
            for (int p = 0; p < KR; ++p)
                if (p < k) {
                    part_s[o + p] = q2_key_score(m[p]);
                    part_i[o + p] = q2_key_entry(m[p]);
                }
        }
    }
}

template <int DT, int RB, int MQ, int KR, int EB>
hipError_t run_qs(const MatchPlan& p, int64_t n, const void* emb, const float* fe, const void* q, const float* fq,
                  int* gthr, int32_t b, int32_t k, float* ps, int* pi, hipStream_t s)
{
    const int work = p.splits * p.qtiles;
    const int grid = work >= 8 ? (work + 7) / 8 * 8 : work;
    k_qs<DT, RB, MQ, KR, EB><<<grid, Q2_NT, 0, s>>>(static_cast<const uint8_t*>(emb), fe, n,
                                                   static_cast<const uint8_t*>(q), fq, gthr, b, k, p.splits,
                                                   p.qtiles, p.b_pad, ps, pi);
    return hipGetLastError();
}

}  // namespace

// shape of the query-stationary kernel: rows of 512, 768, 1024 or 1536 bytes,
// k <= 32.  Lists of 10 slots for k <= 10, 16 for k <= 16 (two query blocks
// per wavefront except for 1536-byte rows), 32 otherwise (one query block).
// Every insertion touches every slot, so the list is kept close to k.
constexpr int q2_kr(int k) { return k <= 10 ? 10 : k <= 16 ? 16 : 32; }
constexpr int q2_mq(int64_t row_bytes, int k) { return k <= 16 && row_bytes != 1536 ? 2 : 1; }
// 32-row blocks per stage and group: four with one query block (two where
// 1536-byte rows and 32-slot lists leave too few registers), two with two
constexpr int q2_eb(int64_t row_bytes, int k)
{
    return q2_mq(row_bytes, k) == 2 || (row_bytes == 1536 && k > 16) ? 2 : 4;
}
constexpr int q2_rows(int64_t row_bytes, int k) { return 32 * q2_eb(row_bytes, k); }
constexpr bool q2_built(int64_t row_bytes, int k)
{
    return (row_bytes == 512 || row_bytes == 768 || row_bytes == 1024 || row_bytes == 1536) && k >= 1 &&
           k <= Q2_KMAX;
}
constexpr int q2_queries(int64_t row_bytes, int k) { return q2_built(row_bytes, k) ? Q2_NW * 32 * q2_mq(row_bytes, k) : 0; }

template <int DT>
hipError_t q2_dispatch(const MatchPlan& p, int64_t n, int64_t rb, const void* emb, const float* fe, const void* q,
                       const float* fq, int* gthr, int32_t b, int32_t k, float* ps, int* pi, hipStream_t s)
{
#define APC_Q2(RB, MQ, KR) run_qs<DT, RB, MQ, KR, q2_eb(RB, KR)>(p, n, emb, fe, q, fq, gthr, b, k, ps, pi, s)
    if (q2_kr(k) == 10) {
        switch (rb) {
        case 1536: return APC_Q2(1536, 1, 10);
        case 1024: return APC_Q2(1024, 2, 10);
        case 768: return APC_Q2(768, 2, 10);
        case 512: return APC_Q2(512, 2, 10);
        }
    } else if (q2_kr(k) == 16) {
        switch (rb) {
        case 1536: return APC_Q2(1536, 1, 16);
        case 1024: return APC_Q2(1024, 2, 16);
        case 768: return APC_Q2(768, 2, 16);
        case 512: return APC_Q2(512, 2, 16);
        }
    } else {
        switch (rb) {
        case 1536: return APC_Q2(1536, 1, 32);
        case 1024: return APC_Q2(1024, 1, 32);
        case 768: return APC_Q2(768, 1, 32);
        case 512: return APC_Q2(512, 1, 32);
        }
    }
#undef APC_Q2
    return hipErrorInvalidValue;
}

hipError_t launch_qs_f16(const MatchPlan& p, int64_t n, int64_t rb, const void* emb, const float* fe, const void* q,
                         const float* fq, int* gthr, int32_t b, int32_t k, float* ps, int* pi, hipStream_t s);
hipError_t launch_qs_bf16(const MatchPlan& p, int64_t n, int64_t rb, const void* emb, const float* fe, const void* q,
                          const float* fq, int* gthr, int32_t b, int32_t k, float* ps, int* pi, hipStream_t s);
hipError_t launch_qs_e4m3(const MatchPlan& p, int64_t n, int64_t rb, const void* emb, const float* fe, const void* q,
                          const float* fq, int* gthr, int32_t b, int32_t k, float* ps, int* pi, hipStream_t s);

}  // namespace apc
