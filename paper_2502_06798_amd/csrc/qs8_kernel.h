// Query-stationary similarity + exact top-k with two wavefronts per SIMD,
// for 16-bit and e4m3 rows of 512, 768 or 1024 bytes (k <= 32), large batches.
//
// Grid: splits x query tiles of 256 queries.  A workgroup of eight
// wavefronts (two per SIMD) owns a query tile and a contiguous range of cache
// entries (its split).  Each wavefront keeps its 32 query rows in VGPRs for
// its whole life, as the B operands of 32x32 MFMAs, in the lane order the
// query preparation writes them (lane l supplies query row l % 32; half
// h = l / 32 supplies bytes [64h, 64h + 64) of every 128-byte chunk of d).
// Cache rows stream through an LDS ring in stages of 64 rows x 256 bytes,
// loaded straight from global memory into LDS; a 16-byte unit of a row sits
// at unit ^ (row % 16), so the A-operand reads (lane = row) are free of bank
// conflicts.  One barrier per stage makes a stage visible to all eight
// wavefronts; each reads every row of it.  Every score is the float32 sum
// over all of d, in the same order whatever the split or tile.
//
// Why two wavefronts per SIMD: the top-k filter is vector-ALU work that one
// wavefront can only issue between its own MFMAs.  Here each wavefront's
// instruction stream mixes the two, and the SIMD interleaves two such
// streams, so the matrix unit keeps busy through the other wavefront's
// filter work and LDS waits.  The price is a register budget of 256 per
// lane: queries (up to 128), two accumulator sets (64), the A fragments of
// two steps (one for 1024-byte rows); the top-k lists therefore live in LDS.
//
// Top-k, per query: one list of k (score, entry) keys in LDS, shared by the
// query's two lanes (they see disjoint rows of each block), unsorted, with
// its fill count and its smallest key and slot held by both lanes.  Groups
// of 64 rows are software-pipelined: while the MFMAs of group g run, the
// same instruction stream scales group g-1's products by their entry factors
// and takes each lane's maximum (the largest score of the lane's 32 pairs,
// exactly: both steps are monotone).  After group g's MFMAs, a lane whose
// maximum reaches its query's filter (the k-th best kept so far; -inf while
// the list has fewer than k) tests its pairs exactly and inserts the ones
// that pass, one per pass: lanes of half 0 first, then half 1, each insert
// replacing the smallest key (or filling an empty slot) and rescanning the
// list for the new smallest.  At the end the list is sorted and written as
// the split's partial list; k_topk_merge merges the splits.
#pragma once

#include "qs_kernel.h"

namespace apc {
namespace {

constexpr int Q8_NW = 8;                        // wavefronts per workgroup (two per SIMD)
constexpr int Q8_NT = Q8_NW * 64;
constexpr int Q8_EB = 2;                        // 32-row blocks per group
constexpr int Q8_GR = Q8_EB * 32;               // rows per group and per stage
constexpr int Q8_STAGE = Q8_GR * Q2_SB;         // bytes of a stage (16 KB)
constexpr int Q8_LPW = Q8_STAGE / 1024 / Q8_NW; // row loads per wavefront per stage
constexpr int Q8_OPS = Q8_LPW + 1;              // vector-memory operations per wavefront per stage
constexpr int Q8_FR = 8;                        // ring of per-group entry factors
constexpr int Q8_KMAX = 32;
constexpr int Q8_QM = 256;                      // groups between refreshes of the quantile bound
constexpr int Q8_QSPLITS = 16;                  // most splits it is shared over

template <int DT, int RB, int KR>
struct Q8Cfg {
    typedef typename Q2Op<DT>::Step Step;
    static constexpr int UPS = Q2Op<DT>::UPS;         // 16-byte units per MFMA step
    static constexpr int SPG = RB / Q2_SB;            // stages per group
    static constexpr int SST = Q2_SB / 32 / UPS;      // MFMA steps per stage
    static constexpr int QST = RB / 32 / UPS;         // steps of a query row held by a lane
    static constexpr int NSTEP = SPG * SST;           // MFMA steps per group
    // steps between an A fragment's read and its MFMA: one for 1024-byte rows,
    // whose 128 VGPRs of queries leave no room for a third fragment set
    static constexpr int LA = RB > 768 ? 1 : 2;
    static constexpr int BQ = Q8_NW * 32;             // queries per workgroup
    static constexpr int LSTR = KR * 8 + 16;          // bytes per query list (padded: no bank conflicts)
    static constexpr int LIST_BYTES = BQ * LSTR;
    static constexpr int SIDE_BYTES = Q8_FR * Q8_GR * 4 + Q8_FR * BQ * 4;
    static constexpr int NS = (Q2_LDS - LIST_BYTES - SIDE_BYTES) / Q8_STAGE;   // stages in the ring
    static_assert(RB == 512 || RB == 768 || RB == 1024, "rows of two to four stages");
    static_assert(NSTEP >= 8, "the filter of a group is spread over eight MFMA steps");
    static_assert(SST >= 3, "fragments are read up to two steps ahead, within the stage for its first steps");
    static_assert(Q8_OPS <= SST - LA + 1, "a stage's loads are issued by the step of its wait for the next stage");
    static_assert(NS >= 4, "LDS ring too small");
    // The entry factors of group g (slot g % FR) are read until the end of
    // group g + 1; the loads of group g + FR start NS - 1 stages early.
    static_assert(SPG * (Q8_FR - 2) >= NS - 1, "entry-factor ring too small");
    static_assert(SPG >= 2, "the shared bounds are loaded with a group's second stage");
    struct Smem {
        uint8_t e[NS * Q8_STAGE];
        float fe[Q8_FR][Q8_GR];
        int gthr[Q8_FR][BQ];                    // shared bounds (keys) seen at a group's second stage
        uint8_t lst[LIST_BYTES];
    };
};

// 16 bytes per lane from global memory straight into LDS, addressed as a
// scalar base plus a per-lane 32-bit offset: lane l's bytes land at lds + 16 l
__device__ inline void q8_dma16(const void* base, uint32_t off, uint32_t lds)
{
    asm volatile("s_nop 0\n\tglobal_load_lds_dwordx4 %0, %1" ::"v"(off), "s"(base), "{m0}"(lds) : "memory");
}

// the same, coherent across the device (values other workgroups update with
// device-scope atomics; a plain load could hit a stale line in this XCD's L2)
__device__ inline void q8_dma16_fresh(const void* base, uint32_t off, uint32_t lds)
{
    asm volatile("s_nop 0\n\tglobal_load_lds_dwordx4 %0, %1 sc1" ::"v"(off), "s"(base), "{m0}"(lds) : "memory");
}

// the value x of the lane 32 apart (lane ^ 32), through the VALU's lane-half
// swap rather than an LDS permute: v_permlane32_swap exchanges lanes 32..63
// of its first operand with lanes 0..31 of its second, so with x in both,
// the second result holds the upper half's x in lanes 0..31 and the first
// the lower half's x in lanes 32..63.  Every lane must be active.
__device__ inline uint32_t q8_partner(uint32_t x, int h)
{
    const auto r = __builtin_amdgcn_permlane32_swap(x, x, false, false);
    return h ? (uint32_t)r[0] : (uint32_t)r[1];
}

// base[off / 4] = v and v = base[off / 4], device-coherent (sc1: written
// through and read past this XCD's L2, so other XCDs' workgroups see them),
// addressed as a wave-uniform base plus a per-lane offset, so that no
// per-lane 64-bit address stays live; the load waits for every vector-memory
// operation in flight (the ring's loads too: they are counted by hand, out of
// the compiler's view)
__device__ inline void q8_store(const int* base, uint32_t off, int v)
{
    asm volatile("global_store_dword %0, %1, %2 sc1" ::"v"(off), "v"(v), "s"(base) : "memory");
}
__device__ inline int q8_load_now(const int* base, uint32_t off)
{
    int v;
    asm volatile("global_load_dword %0, %1, %2 sc1\n\ts_waitcnt vmcnt(0)" : "=v"(v) : "v"(off), "s"(base) : "memory");
    return v;
}
// device-scope signed max of v into base[off / 4]
__device__ inline void q8_atomic_max(const int* base, uint32_t off, int v)
{
    asm volatile("global_atomic_smax %0, %1, %2" ::"v"(off), "v"(v), "s"(base) : "memory");
}

template <int DT, int RB, int KR>
__global__ __launch_bounds__(Q8_NT) void k_qs8(
    const uint8_t* __restrict__ emb, const float* __restrict__ fe, int64_t n,
    const uint8_t* __restrict__ qry, const float* __restrict__ fq_ws, int* __restrict__ gthr, int* __restrict__ g2, int32_t b,
    int32_t k, int splits, int qtiles, float* __restrict__ part_s, int* __restrict__ part_i)
{
    typedef Q8Cfg<DT, RB, KR> C;
    typedef typename C::Step Step;
    constexpr int NS = C::NS, SPG = C::SPG, SST = C::SST, UPS = C::UPS, NSTEP = C::NSTEP;
    constexpr int RPW = Q8_GR / Q8_NW;                             // rows of a stage each wavefront loads
    __shared__ typename C::Smem sm;
    const int tid = threadIdx.x, lane = tid & 63, h = lane >> 5, r32 = lane & 31;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);

    // workgroup id -> (split, query tile): with a grid that is a multiple of 8,
    // consecutive linear ids share an XCD (workgroups are dealt round-robin
    // over the 8 XCDs), so the query tiles of a split share its L2
    const int grid = (int)gridDim.x, work = splits * qtiles;
    const int lin = (grid & 7) == 0 ? (int)(blockIdx.x & 7) * (grid >> 3) + (int)(blockIdx.x >> 3) : (int)blockIdx.x;
    if (lin >= work) return;                                       // whole workgroup: uniform
    const int split = lin / qtiles, qtile = lin % qtiles;
    const int64_t q0w = (int64_t)qtile * C::BQ + wave * 32;       // this wavefront's first query

    const int64_t ngr = (n + Q8_GR - 1) / Q8_GR;                   // groups of the cache
    const int64_t g_begin = ngr * split / splits;
    const int ng = (int)(ngr * (split + 1) / splits - g_begin);   // groups of this split (>= 1)

    // ---- queries into VGPRs (in load order), the query factor.  Wavefronts
    // past the batch compute on the zero padding of the query copy; their
    // factor is NaN, so nothing of theirs is kept ----
    Step qv[C::QST];
    {
        const uint8_t* qblk = qry + (((int64_t)qtile * Q8_NW + wave) * C::QST * 64 + lane) * sizeof(Step);
#pragma unroll
        for (int s = 0; s < C::QST; ++s) qv[s] = *reinterpret_cast<const Step*>(qblk + (int64_t)s * 64 * sizeof(Step));
    }
    const float fq = fq_ws[q0w + r32];
    // 1 / fq for the exact test's threshold (1024-byte rows: no register to
    // spare, the threshold divides)
    const float rfq = RB == 1024 ? 0.f : 1.0f / fq;
    // wait for these loads here: inside the loop the compiler's own waits
    // would also drain the ring's loads, which it does not see
#pragma unroll
    for (int s = 0; s < C::QST; ++s) q2_use(qv[s]);
    asm volatile("" ::"v"(fq));

    // ---- stage loads.  Wavefront w fills rows [RPW w, RPW (w + 1)) of a
    // stage.  One more load per stage: at a group's second stage, lanes 0..7
    // bring the shared bounds of the wavefront's 32 queries (as late as the
    // ring allows, so they include what other workgroups published
    // meanwhile); at its other stages lanes 0..15 bring the group's 64 entry
    // factors (the same bytes each time).  So every stage is Q8_OPS vector-
    // memory operations per wavefront.  Stages past the split repeat the
    // split's last stage into their (unused) ring slot, which keeps the
    // counts of every wait the same. ----
    const uint32_t lds_e = (uint32_t)(size_t)(lds_void*)sm.e;
    const uint32_t lds_fe = (uint32_t)(size_t)(lds_void*)&sm.fe[0][0];
    const uint32_t lds_gt = (uint32_t)(size_t)(lds_void*)&sm.gthr[0][0];
    // load i of a wavefront: row wave RPW + 4 i + lane / 16 of the stage, the
    // logical unit (lane % 16) ^ (row % 16) of it stored at unit lane % 16
    auto lrow = [&](int i) __attribute__((always_inline)) { return wave * RPW + i * 4 + (lane >> 4); };
    auto loff = [&](int i) __attribute__((always_inline)) { return (uint32_t)(((lane & 15) ^ (lrow(i) & 15)) * 16); };
    // (load 1's row is load 0's + 4, whose low four bits differ in bit 2
    // only: its unit offset is load 0's ^ 64, and RB is a multiple of 256)
    static_assert(Q8_LPW == 2, "two row loads per wavefront and stage");
    const uint32_t voff0 = (uint32_t)lrow(0) * RB + loff(0);
    // Stage gi SPG + D of the schedule, D a compile-time offset, for group gi
    // whose first row is at gbase, whose entry factors are at fbase and whose
    // first stage uses ring slot gslot (all kept up to date by the group loop,
    // so the addresses of a group inside the split take a few scalar
    // additions; only the split's last group and the stages past it take the
    // general path).
    const int64_t grp_bytes = (int64_t)Q8_GR * RB;
    const uint8_t* const last_base = emb + (g_begin + ng - 1) * grp_bytes + (SPG - 1) * Q2_SB;   // the split's last stage
    const int64_t tail = n - (g_begin + ng - 1) * Q8_GR;          // rows of the split's last group (<= 64)
    // Part P < Q8_LPW is row load P, part Q8_LPW the side load; a part
    // outside [0, Q8_OPS) issues all of them.
    auto issue = [&](int gi, const uint8_t* gbase, const float* fbase, int gslot, auto dc, auto pc)
                     __attribute__((always_inline)) {
        constexpr int D = decltype(dc)::value, DG = D / SPG, JJ = D % SPG, P = decltype(pc)::value;
        constexpr bool all = P < 0 || P >= Q8_OPS;
        auto row_part = [&](int i) __attribute__((always_inline)) { return all || P == i; };
        constexpr bool side_part = all || P == Q8_LPW;
        const int g = gi + DG;                                     // the stage's group
        int slot = gslot + D % NS;                                 // (gslot + D) mod NS, gslot < NS
        if (slot >= NS) slot -= NS;
        const uint32_t m0 = lds_e + (uint32_t)slot * Q8_STAGE + (uint32_t)(wave * RPW) * Q2_SB;
        const uint32_t soff = (uint32_t)lane * 16;                 // lanes past the side data idle
        // the side load of group gq into its ring slot
        auto side = [&](int gq, const float* fg) __attribute__((always_inline)) {
            if constexpr (!side_part) return;
            if constexpr (JJ == 1) {
                if (lane < 8)
                    q8_dma16_fresh(gthr + q0w, soff, lds_gt + (uint32_t)(((gq & (Q8_FR - 1)) * C::BQ + wave * 32) * 4));
            } else {
                if (lane < Q8_GR / 4) q8_dma16(fg, soff, lds_fe + (uint32_t)(gq & (Q8_FR - 1)) * (Q8_GR * 4));
            }
        };
        if (g < ng - 1) {
            // a whole group inside the split: constant offsets from the running bases
            const uint8_t* base = gbase + DG * grp_bytes + JJ * Q2_SB;
#pragma unroll
            for (int i = 0; i < Q8_LPW; ++i)
                if (row_part(i)) q8_dma16(base, i ? (voff0 ^ 64u) + 4 * RB : voff0, m0 + i * 4 * Q2_SB);
            side(g, fbase + DG * Q8_GR);
        } else {
            // the split's last group (its rows past the cache repeat its last
            // row), or past the split (a repeat of its last stage)
            const bool past = g >= ng;
            const uint8_t* base = past ? last_base : gbase + DG * grp_bytes + JJ * Q2_SB;
            if (tail == Q8_GR) {
#pragma unroll
                for (int i = 0; i < Q8_LPW; ++i)
                    if (row_part(i)) q8_dma16(base, i ? (voff0 ^ 64u) + 4 * RB : voff0, m0 + i * 4 * Q2_SB);
            } else {
                const int last = (int)tail - 1;                    // last valid row of the group
#pragma unroll
                for (int i = 0; i < Q8_LPW; ++i)
                    if (row_part(i))
                        q8_dma16(base, (uint32_t)(lrow(i) < last ? lrow(i) : last) * RB + loff(i), m0 + i * 4 * Q2_SB);
            }
            side(ng - 1, fe + (g_begin + ng - 1) * Q8_GR);
        }
    };
    // wait until stage u has landed (this wavefront's loads; stages up to
    // u + NS - 2 have been issued), then make it visible to every wavefront
    auto wait_stage = [&]() __attribute__((always_inline)) {
        __builtin_amdgcn_s_waitcnt(q2_vmcnt((NS - 2) * Q8_OPS));
        __syncthreads();
    };
    static_for<NS - 1>([&](auto dc) __attribute__((always_inline)) {
        issue(0, emb + g_begin * grp_bytes, fe + g_begin * Q8_GR, 0, dc, std::integral_constant<int, -1>{});
    });

    // ---- list state of this lane's query.  The list's slots are split
    // between the two lanes by pairs (slots 2p, 2p + 1 belong to half p % 2);
    // each lane knows the smallest key of its own slots, and both know the
    // fill count and the smallest key of the whole list and its slot ----
    // (every access of a list goes through uint64_t, so that the compiler
    // keeps a lane's stores and its partner's later loads in order)
    uint64_t* const lst = reinterpret_cast<uint64_t*>(sm.lst + (wave * 32 + r32) * C::LSTR);
    // slots from k on (this lane's) hold the largest key, for the rescans
#pragma unroll
    for (int i = 0; i < KR / 2; ++i) {
        const int sl = 2 * h + 4 * (i >> 1) + (i & 1);
        if (sl >= k) lst[sl] = ~0ull;
    }
    int cnt = 0;                 // keys in the list
    uint64_t wkey = 0;           // its smallest key (valid once cnt == k)
    int wslot = 0;               // and that key's slot
    float own = neg_inf();       // the list's k-th best score (-inf while cnt < k)
    uint64_t hkey = ~0ull;       // the smallest key of this lane's slots
    int hslot = 0;               // and its slot
    // the smallest of this lane's keys and its slot (slots from k on hold the
    // largest key, so they are never the smallest of a full list): its KR / 2
    // slots read eight at a time, each eight through a tree of comparisons;
    // for 1024-byte rows, whose registers are full, in a loop over the first k
    auto rescan = [&]() __attribute__((always_inline)) {
        if constexpr (RB == 1024) {
            uint64_t best = ~0ull;
            int bs = 0;
#pragma unroll 1
            for (int c0 = 2 * h; c0 < k; c0 += 16) {               // slots c0 + 4 i, + 1: this half's
                uint64_t v[8];
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    v[2 * i] = lst[c0 + 4 * i];
                    v[2 * i + 1] = lst[c0 + 4 * i + 1];
                }
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const uint64_t k0 = v[2 * i], k1 = v[2 * i + 1];
                    const int p0 = c0 + 4 * i;
                    if (p0 < k && k0 < best) { best = k0; bs = p0; }
                    if (p0 + 1 < k && k1 < best) { best = k1; bs = p0 + 1; }
                }
            }
            hkey = best;
            hslot = bs;
        } else {
            constexpr int HS = KR / 2, CH = HS < 8 ? HS : 8;
            uint64_t best = ~0ull;
            int bs = 0;
#pragma unroll 1
            for (int c0 = 0; c0 < HS; c0 += CH) {
                uint64_t v[CH];
                int vs[CH];
#pragma unroll
                for (int i = 0; i < CH; ++i) {
                    vs[i] = 2 * h + 4 * ((c0 + i) >> 1) + ((c0 + i) & 1);   // this half's slots
                    v[i] = lst[vs[i]];
                }
#pragma unroll
                for (int w = 1; w < CH; w *= 2)
#pragma unroll
                    for (int i = 0; i + w < CH; i += 2 * w) {
                        const bool tk = v[i + w] < v[i];
                        v[i] = tk ? v[i + w] : v[i];
                        vs[i] = tk ? vs[i + w] : vs[i];
                    }
                const bool tk = v[0] < best;
                best = tk ? v[0] : best;
                bs = tk ? vs[0] : bs;
            }
            hkey = best;
            hslot = bs;
        }
    };
    // the list's smallest key and slot from both lanes' (all lanes take part)
    auto combine = [&]() __attribute__((always_inline)) {
        const uint32_t olo = q8_partner((uint32_t)hkey, h), ohi = q8_partner((uint32_t)(hkey >> 32), h);
        const int os = (int)q8_partner((uint32_t)hslot, h);
        const uint64_t ob = ((uint64_t)ohi << 32) | olo;
        wkey = ob < hkey ? ob : hkey;
        wslot = ob < hkey ? os : hslot;
        own = cnt >= k ? q2_key_score(wkey) : neg_inf();
    };

    // one piece of the filter of the previous group (four of a lane's values,
    // scaled in place by their entry factors; m takes their maximum)
    auto filter_piece = [&](auto pc, f32x16 (&prv)[Q8_EB], const float* frp, float& m) __attribute__((always_inline)) {
        constexpr int P = decltype(pc)::value;
        constexpr int eb = P / 4, g4 = P % 4;
        const float4 f4 = *reinterpret_cast<const float4*>(frp + eb * 32 + 8 * g4 + 4 * h);
        const float fv[4] = {f4.x, f4.y, f4.z, f4.w};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            float x = prv[eb][4 * g4 + i] * fv[i];
            asm volatile("" : "+v"(x));                            // computed here, between the MFMAs,
            prv[eb][4 * g4 + i] = x;                               // not sunk to where it is used
            m = __builtin_fmaxf(m, x);
        }
        asm volatile("" : "+v"(m));
    };

    // the exact test and the insertions of group gp, whose products times
    // entry factors are in prv and whose lane maxima are m.  The filter F is
    // the largest known lower bound on the query's k-th best score: the k-th
    // of this split's list, or the shared bound G (the largest k-th of any
    // split's list published so far, read from slot gs: k entries score at
    // least that much; ties with it are kept).
    auto finish = [&](int gp, int gs, f32x16 (&prv)[Q8_EB], float m) __attribute__((always_inline)) {
        const float G = q2_unkey(sm.gthr[gs & (Q8_FR - 1)][wave * 32 + r32]);
        const float F = __builtin_fmaxf(own, G);
        const bool pass = fq == fq && clamp1(m * fq) >= F;         // NaN f_q: row not matched
        if (!__builtin_amdgcn_ballot_w64(pass)) return;
        const int64_t e0 = (g_begin + gp) * Q8_GR;
        uint32_t mask = 0;
        if (pass) {
            if (F <= -1.f) {
                mask = ~0u;
            } else {
                // the pairs whose score can reach F: y fq >= F implies y >= Fy,
                // Fy = F / fq moved away from zero by far more than the rounding
                // of either side (F times the rounded 1 / fq is within 2^-23 of
                // F / fq, relative; the margin is 2^-18).  This admits a few
                // more pairs than the exact test; each is then kept only if its
                // exact key beats the list's smallest, so the list is unchanged
                // by the extras.
                const float fy = RB == 1024 ? F / fq : F * rfq;
                const float Fy = fy > 0.f ? fy * (1.f - 0x1p-18f) : fy * (1.f + 0x1p-18f);
#pragma unroll
                for (int j = 31; j >= 0; --j) mask = q2_shift_in(mask, prv[j >> 4][j & 15] >= Fy);
            }
            if (e0 + Q8_GR > n) {
                // rows past the cache: the lane's rows 32 eb + 8 g + 4 h + i,
                // value 16 eb + 4 g + i, grow with the value index, so the valid
                // values are a prefix (of length c_h, from scalar arithmetic)
                const int64_t rem = n - e0;                        // valid rows of the group, < 64
                int c0 = 0, c1 = 0;
#pragma unroll
                for (int el = 0; el < 32; ++el) {
                    const int row = 32 * (el >> 4) + 8 * ((el & 15) >> 2) + (el & 3);
                    c0 += row < rem;
                    c1 += row + 4 < rem;
                }
                const int c = h ? c1 : c0;
                mask &= c >= 32 ? ~0u : (1u << c) - 1u;
            }
        }
#pragma unroll
        for (int hh = 0; hh < 2; ++hh) {
            while (__builtin_amdgcn_ballot_w64(h == hh && mask != 0)) {
                const bool act = h == hh && mask != 0;
                const int bsel = act ? __builtin_ctz(mask) : 0;
                if (act) mask &= mask - 1;
                const float sc = clamp1(q2_pick<Q8_EB>(prv, bsel) * fq);
                const int r = bsel & 15;
                const int e = (int)(e0 + 32 * (bsel >> 4) + 8 * (r >> 2) + 4 * h + (r & 3));
                const uint64_t key = q2_pack(sc, e);
                const bool ins = act && (cnt < k || key > wkey);
                if (ins) lst[cnt < k ? cnt : wslot] = key;
                // both lanes of the query follow the inserting one (every lane
                // takes part in the exchange: a lane whose partner is masked
                // off would read 0)
                const uint32_t pins = q8_partner((uint32_t)ins, h);
                const bool did = h == hh ? ins : pins != 0u;
                if (did) {
                    if (cnt < k) ++cnt;
                    if (cnt == k) rescan();
                }
                combine();
            }
        }
        // publish this split's k-th best when it beats the shared bound
        if (h == 0 && own > G) q8_atomic_max(gthr + q0w, (uint32_t)r32 * 4, q2_key(own));
    };

    // A second bound, shared through the same slot.  Split s publishes, per
    // query, a score v_s that at least r = ceil(k / splits) keys of its list
    // reach: the smaller of its two halves' ceil(r / 2)-th largest (the
    // larger of the two maxima when r = 1).  The splits' rows are disjoint,
    // so at least splits * r >= k keys reach min_s v_s: a lower bound on the
    // query's k-th best, whatever each split's progress (a list only
    // improves, so an old v_s stays valid).  For splits of equal progress it
    // is about the k-th best of all their rows together, where each split's
    // own k-th is that of a quarter of them (with four splits).  It is
    // refreshed every Q8_QM groups: a scan of the list, one store, and one
    // load per split.
    const int64_t b_pad = (int64_t)qtiles * C::BQ;
    auto share_quantile = [&]() __attribute__((always_inline)) {
        const int rq = (k + splits - 1) / splits, rh = (rq + 1) / 2;
        // this lane's slots' rh-th largest order word (the key's upper 32
        // bits; counting equal words; 0 if the half holds fewer), by rh
        // passes over the slots, each finding the largest word below the
        // previous pass's and how often it occurs
        constexpr int HS = KR / 2;
        const uint32_t* const lw = reinterpret_cast<const uint32_t*>(lst);   // word 2 c + 1: slot c's order word
        uint32_t prev = ~0u, u = 0u;
        int need = rh;
        bool found = false;
#pragma unroll 1
        for (int it = 0; it < rh; ++it) {
            asm volatile("" ::: "memory");                         // read the slots again: no copy held in registers
            uint32_t mx = 0u;
            int c = 0;
#pragma unroll 2
            for (int i = 0; i < HS; ++i) {
                const int sl = 2 * h + 4 * (i >> 1) + (i & 1);     // this half's slots
                uint32_t x = sl < cnt ? lw[2 * sl + 1] : 0u;
                x = x < prev ? x : 0u;
                c = x > mx ? 1 : c + (x == mx ? 1 : 0);
                mx = x > mx ? x : mx;
            }
            if (!found && mx != 0u) {
                if (c >= need) {
                    u = mx;
                    found = true;
                } else {
                    need -= c;
                    prev = mx;
                }
            }
        }
        const uint32_t uo = q8_partner(u, h);
        const uint32_t v = rq <= 1 ? __builtin_elementwise_max(u, uo) : __builtin_elementwise_min(u, uo);
        const int key = q2_key(q2_key_score((uint64_t)v << 32));  // -inf for 0
        if (h == 0) {
            const uint32_t off = (uint32_t)r32 * 4;
            q8_store(g2 + split * b_pad + q0w, off, key);
            int mn = key;
            for (int sp = 0; sp < splits; ++sp) mn = __builtin_elementwise_min(mn, q8_load_now(g2 + sp * b_pad + q0w, off));
            if (mn > q2_key(neg_inf())) q8_atomic_max(gthr + q0w, off, mn);
        }
    };

    // A fragments: the per-lane byte offset (row and swizzled unit) of the
    // first unit a step of a stage reads, fixed for the kernel; block eb
    // adds eb 8 KB.  An e4m3 step's second unit is logical unit lu + 1 (lu
    // even), stored at unit (lu ^ x) ^ 1: its offset is the first's ^ 16
    // (stage and row offsets are multiples of 256).
    // Step ss reads logical unit lu = 4 h + c (c = 8 cl + sp has no bit in
    // common with 4 h), stored at unit lu ^ (r32 % 16) = (4 h ^ (r32 % 16)) ^ c:
    // one offset per lane, uo0, and a constant per step.
    const uint32_t uo0 = (uint32_t)(r32 * Q2_SB + (((h * 4) ^ (r32 & 15)) * 16));
    auto uo = [&](int ss) __attribute__((always_inline)) {
        const int cl = ss / (4 / UPS), sp = (ss % (4 / UPS)) * UPS;
        return uo0 ^ (uint32_t)((cl * 8 + sp) * 16);
    };
    auto rd = [&](const uint8_t* sbase, int ss, Step (&dst)[Q8_EB]) __attribute__((always_inline)) {
        const uint32_t base = (uint32_t)(size_t)(lds_void*)sbase;
        const uint32_t a0 = base + uo(ss);
#pragma unroll
        for (int eb = 0; eb < Q8_EB; ++eb) {
            const uint8_t* rp = sbase + eb * 32 * Q2_SB;
            if constexpr (UPS == 1) {
                dst[eb] = *reinterpret_cast<const uint4*>(rp + uo(ss));
            } else {
                const uint4 x0 = *reinterpret_cast<const uint4*>(rp + uo(ss));
                const uint4 x1 = *reinterpret_cast<const uint4*>(rp + ((a0 ^ 16u) - base));
                dst[eb] = Step{(int)x0.x, (int)x0.y, (int)x0.z, (int)x0.w, (int)x1.x, (int)x1.y, (int)x1.z, (int)x1.w};
            }
        }
    };

    // group gi: its MFMAs into acc; the filter of group gi - 1 (in prv) spread
    // over them; then the exact test and insertions of group gi - 1.  The A
    // fragments are read LA steps ahead of their MFMAs.  The wait and
    // barrier for a stage's successor come LA steps before the stage's end,
    // so the successor's first fragments are read while the stage's last
    // MFMAs run (the barrier follows all reads of the stage: the slot may
    // then be refilled).  For gi = 0, prv holds zeros and nothing is tested.
    auto group = [&](int gi, const uint8_t* gbase, const float* fbase, int gslot, f32x16 (&acc)[Q8_EB],
                     f32x16 (&prv)[Q8_EB])
                     __attribute__((always_inline)) {
        const float* frp = sm.fe[(gi - 1) & (Q8_FR - 1)];
        float m = neg_inf();
        Step a0[Q8_EB], a1[Q8_EB], a2[Q8_EB];
        static_for<SPG>([&](auto jc) __attribute__((always_inline)) {
            constexpr int j = decltype(jc)::value;
            int sl = gslot + j % NS, sln = gslot + (j + 1) % NS;  // ring slots of stages t, t + 1
            if (sl >= NS) sl -= NS;
            if (sln >= NS) sln -= NS;
            const uint8_t* sb = sm.e + sl * Q8_STAGE;
            const uint8_t* sbn = sm.e + sln * Q8_STAGE;
            if constexpr (j == 0) {
                wait_stage();
                rd(sb, 0, a0);
                if constexpr (C::LA == 2) rd(sb, 1, a1);
            }
            static_for<SST>([&](auto sc) __attribute__((always_inline)) {
                constexpr int ss = decltype(sc)::value;
                constexpr int st = j * SST + ss;                   // MFMA step of the group
                constexpr int tg = ss + C::LA;                     // step whose fragments are read now
                Step (&an)[Q8_EB] = C::LA == 2 ? a2 : a1;          // where they go
                // the stage's loads into the slot stage t - 1 used, one per
                // step (all before the wait at step SST - 2, whose count
                // includes them), so that the workgroup's loads are not one
                // burst after the barrier
                if constexpr (ss < Q8_OPS)
                    issue(gi, gbase, fbase, gslot, std::integral_constant<int, j + NS - 1>{}, std::integral_constant<int, ss>{});
                if constexpr (tg < SST) {
                    rd(sb, tg, an);
                } else if constexpr (j + 1 < SPG) {
                    if constexpr (tg == SST) wait_stage();
                    rd(sbn, tg - SST, an);
                }
#pragma unroll
                for (int eb = 0; eb < Q8_EB; ++eb) q2_mma<DT>(acc[eb], a0[eb], qv[st], st == 0);
                // filter piece P of the previous group at step floor(P NSTEP / 8)
                static_for<8>([&](auto pc) __attribute__((always_inline)) {
                    if constexpr (decltype(pc)::value * NSTEP / 8 == st) filter_piece(pc, prv, frp, m);
                });
#pragma unroll
                for (int eb = 0; eb < Q8_EB; ++eb) {
                    a0[eb] = a1[eb];
                    if constexpr (C::LA == 2) a1[eb] = a2[eb];
                }
                __builtin_amdgcn_sched_barrier(0);
            });
        });
        if (gi >= 1) finish(gi - 1, gi, prv, m);
        if ((gi & (Q8_QM - 1)) == Q8_QM - 1 && splits > 1 && splits <= Q8_QSPLITS) share_quantile();
    };

    f32x16 acc0[Q8_EB], acc1[Q8_EB];
#pragma unroll
    for (int eb = 0; eb < Q8_EB; ++eb) {
        acc0[eb] = f32x16{};
        acc1[eb] = f32x16{};
    }
    const uint8_t* gbase = emb + g_begin * grp_bytes;
    const float* fbase = fe + g_begin * Q8_GR;
    int gslot = 0;
    auto next_group = [&]() __attribute__((always_inline)) {
        gbase += grp_bytes;
        fbase += Q8_GR;
        gslot += SPG % NS;                                         // correct also if a group spans more stages than the ring
        if (gslot >= NS) gslot -= NS;
    };
    for (int gi = 0; gi < ng; gi += 2) {
        group(gi, gbase, fbase, gslot, acc0, acc1);
        next_group();
        if (gi + 1 < ng) {
            group(gi + 1, gbase, fbase, gslot, acc1, acc0);
            next_group();
        }
    }
    __builtin_amdgcn_s_waitcnt(q2_vmcnt(0));                       // the loads past the split
    if (q0w >= b) return;
    // the last group's filter and insertions
    {
        const int gl = ng - 1;
        const float* frp = sm.fe[gl & (Q8_FR - 1)];
        float m = neg_inf();
        auto drain = [&](f32x16 (&last)[Q8_EB]) __attribute__((always_inline)) {
            static_for<8>([&](auto pc) __attribute__((always_inline)) { filter_piece(pc, last, frp, m); });
            finish(gl, gl, last, m);
        };
        if (gl & 1) drain(acc1);
        else drain(acc0);
    }

    // ---- the split's partial list: sorted, the k best (empty slots last) ----
    const int64_t qg = q0w + r32;
    if (h == 0) {
        constexpr int KP = KR <= 16 ? 16 : 32;
        uint64_t x[KP];
#pragma unroll
        for (int p = 0; p < KP; ++p) x[p] = p < cnt ? lst[p] : 0ull;
        // bitonic sort, descending
#pragma unroll
        for (int size = 2; size <= KP; size *= 2)
#pragma unroll
            for (int stride = size / 2; stride > 0; stride /= 2)
#pragma unroll
                for (int i = 0; i < KP; ++i) {
                    const int jx = i ^ stride;
                    if (jx > i) {
                        const bool desc = (i & size) == 0;
                        const bool sw = desc ? x[i] < x[jx] : x[i] > x[jx];
                        const uint64_t a0 = x[i], a1 = x[jx];
                        x[i] = sw ? a1 : a0;
                        x[jx] = sw ? a0 : a1;
                    }
                }
        const int64_t o = (qg * splits + split) * k;
#pragma unroll
        for (int p = 0; p < KR; ++p)
            if (p < k) {
                part_s[o + p] = q2_key_score(x[p]);
                part_i[o + p] = q2_key_entry(x[p]);
            }
    }
}

template <int DT, int RB, int KR>
hipError_t run_qs8(const MatchPlan& p, int64_t n, const void* emb, const float* fe, const void* q, const float* fq,
                   int* gthr, int* g2, int32_t b, int32_t k, float* ps, int* pi, hipStream_t s)
{
    const int work = p.splits * p.qtiles;
    const int grid = work >= 8 ? (work + 7) / 8 * 8 : work;
    k_qs8<DT, RB, KR><<<grid, Q8_NT, 0, s>>>(static_cast<const uint8_t*>(emb), fe, n, static_cast<const uint8_t*>(q),
                                              fq, gthr, g2, b, k, p.splits, p.qtiles, ps, pi);
    return hipGetLastError();
}

}  // namespace

constexpr bool q8_built(int64_t row_bytes, int k)
{
    return (row_bytes == 512 || row_bytes == 768 || row_bytes == 1024) && k >= 1 && k <= Q8_KMAX;
}

template <int DT>
hipError_t q8_dispatch(const MatchPlan& p, int64_t n, int64_t rb, const void* emb, const float* fe, const void* q,
                       const float* fq, int* gthr, int* g2, int32_t b, int32_t k, float* ps, int* pi, hipStream_t s)
{
    if (k <= 16) {
        if (rb == 1024) return run_qs8<DT, 1024, 16>(p, n, emb, fe, q, fq, gthr, g2, b, k, ps, pi, s);
        if (rb == 768) return run_qs8<DT, 768, 16>(p, n, emb, fe, q, fq, gthr, g2, b, k, ps, pi, s);
        if (rb == 512) return run_qs8<DT, 512, 16>(p, n, emb, fe, q, fq, gthr, g2, b, k, ps, pi, s);
    } else if (k <= Q8_KMAX) {
        if (rb == 1024) return run_qs8<DT, 1024, 32>(p, n, emb, fe, q, fq, gthr, g2, b, k, ps, pi, s);
        if (rb == 768) return run_qs8<DT, 768, 32>(p, n, emb, fe, q, fq, gthr, g2, b, k, ps, pi, s);
        if (rb == 512) return run_qs8<DT, 512, 32>(p, n, emb, fe, q, fq, gthr, g2, b, k, ps, pi, s);
    }
    return hipErrorInvalidValue;
}

hipError_t launch_qs8_f16(const MatchPlan& p, int64_t n, int64_t rb, const void* emb, const float* fe, const void* q,
                          const float* fq, int* gthr, int* g2, int32_t b, int32_t k, float* ps, int* pi, hipStream_t s);
hipError_t launch_qs8_bf16(const MatchPlan& p, int64_t n, int64_t rb, const void* emb, const float* fe, const void* q,
                           const float* fq, int* gthr, int* g2, int32_t b, int32_t k, float* ps, int* pi, hipStream_t s);
hipError_t launch_qs8_e4m3(const MatchPlan& p, int64_t n, int64_t rb, const void* emb, const float* fe, const void* q,
                           const float* fq, int* gthr, int* g2, int32_t b, int32_t k, float* ps, int* pi, hipStream_t s);

}  // namespace apc
