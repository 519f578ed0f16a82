// Optimal level and capacity-constrained placement of a batch of queries.
//
// One workgroup of 1024 threads.  The level of query q is the number of
// thresholds at or below its best score.  Placement runs rounds r = 0..L:
// every unassigned query applies to the r-th entry of its preference list
// [lam, lam-1, .., 0, lam+1, .., L]; a level accepts applicants in query
// order while it has places left.  Within a round, levels do not interact,
// so each 1024-query chunk computes every applicant's rank among the
// applicants of its level with one wave ballot per level (prefix counts in
// lane order) plus per-wave totals summed in wave order; chunks run in
// query order.  Ranks therefore never depend on atomic ordering, and the
// result is deterministic.  A placement of rank t at level p lands on the
// level's instances ordered by (queue desc, index asc), each filled up to
// its capacity.
#include "apc_internal.h"
#include "route_plan.h"

namespace apc {
namespace {

constexpr int NT = 1024;
constexpr int NWAVE = NT / 64;

// The table is a kernel argument.  Kernel-argument memory is read through
// uncached paths, so every per-lane (dynamically indexed) read of it would be
// a full memory round trip; the kernels copy it into LDS once instead.
// All of a thread's loads are issued before its stores: one round trip.
static_assert(sizeof(AssignTable) % 4 == 0, "table copied as 32-bit words");
template <int NTHR>
__device__ inline void table_to_lds(const AssignTable& src, AssignTable& dst, int tid)
{
    constexpr int W = (int)(sizeof(AssignTable) / 4), PER = (W + NTHR - 1) / NTHR;
    const uint32_t* s = reinterpret_cast<const uint32_t*>(&src);
    uint32_t* d = reinterpret_cast<uint32_t*>(&dst);
    uint32_t v[PER];
#pragma unroll
    for (int i = 0; i < PER; ++i) v[i] = tid + i * NTHR < W ? s[tid + i * NTHR] : 0u;
#pragma unroll
    for (int i = 0; i < PER; ++i)
        if (tid + i * NTHR < W) d[tid + i * NTHR] = v[i];
    __syncthreads();
}

__global__ __launch_bounds__(NT) void k_assign(const AssignTable targ, const float* __restrict__ top_score,
                                                int32_t ld, int32_t b, int32_t* __restrict__ opt_level,
                                                int32_t* __restrict__ out_level,
                                                int32_t* __restrict__ out_inst,
                                                int32_t* __restrict__ out_slot,
                                                int32_t* __restrict__ inst_fill)
{
    __shared__ int used[APC_MAX_LEVELS + 1];
    __shared__ int wcnt[NWAVE][APC_MAX_LEVELS + 1];
    __shared__ AssignTable t;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    table_to_lds<NT>(targ, t, tid);
    const int L = t.L;
    const uint64_t lt_mask = (lane == 0) ? 0ull : (~0ull >> (64 - lane));

    for (int q = tid; q < b; q += NT) {
        const float best = top_score[(int64_t)q * ld];
        int lam = 0;
        for (int l = 0; l < L; ++l) lam += best >= t.theta[l];
        opt_level[q] = lam;
        out_level[q] = -1;
        out_slot[q] = -1;
    }
    if (tid <= L) used[tid] = 0;
    __syncthreads();

    for (int r = 0; r <= L; ++r) {
        for (int base = 0; base < b; base += NT) {
            const int q = base + tid;
            int want = -1;
            if (q < b && out_level[q] < 0) {
                const int lam = opt_level[q];
                want = r <= lam ? lam - r : r;
            }
            int pre = 0;
            for (int p = 0; p <= L; ++p) {
                const uint64_t m = __ballot(want == p);
                if (want == p) pre = __popcll(m & lt_mask);
                if (lane == 0) wcnt[wave][p] = __popcll(m);
            }
            __syncthreads();
            if (want >= 0) {
                int rank = used[want] + pre;
                for (int w = 0; w < wave; ++w) rank += wcnt[w][want];
                if (rank < t.level_cap[want]) {
                    out_level[q] = want;
                    out_slot[q] = rank;           // admission rank until the instance pass below
                }
            }
            __syncthreads();
            if (tid <= L) {
                int tot = 0;
                for (int w = 0; w < NWAVE; ++w) tot += wcnt[w][tid];
                const int u = used[tid] + tot;
                used[tid] = u < t.level_cap[tid] ? u : t.level_cap[tid];
            }
            __syncthreads();
        }
    }

    for (int q = tid; q < b; q += NT) {
        const int p = out_level[q];
        int inst = -1, slot = -1;
        if (p >= 0) {
            const int rank = out_slot[q];
            for (int j = t.level_first[p]; j < t.level_first[p + 1]; ++j)
                if (rank < t.ord_cum[j] + t.ord_cap[j]) {
                    inst = t.ord_inst[j];
                    slot = rank - t.ord_cum[j];
                    break;
                }
        }
        out_inst[q] = inst;
        out_slot[q] = slot;
    }
    for (int p = 0; p <= L; ++p)
        for (int j = t.level_first[p] + tid; j < t.level_first[p + 1]; j += NT) {
            int f = used[p] - t.ord_cum[j];
            f = f < 0 ? 0 : (f > t.ord_cap[j] ? t.ord_cap[j] : f);
            inst_fill[t.ord_inst[j]] = f;
        }
}

// The same with every query's state in registers (thread tid owns queries
// tid + c NTB, c < QPT): no global-memory round trip per round.  The block
// is sized to the batch (NTB threads).  Each chunk of a round takes two
// barriers: after the per-wave ballots, and after the ranks, which read the
// level counts of the round so far (used[cur]) while threads p <= L write the
// counts after this chunk into the other buffer.  The rounds stop once a round
// has no applicant (every query placed; later rounds would change nothing).
template <int QPT, int NTB>
__global__ __launch_bounds__(NTB) void k_assign_reg(const AssignTable targ, const float* __restrict__ top_score,
                                                    int32_t ld, int32_t b, int32_t* __restrict__ opt_level,
                                                    int32_t* __restrict__ out_level,
                                                    int32_t* __restrict__ out_inst,
                                                    int32_t* __restrict__ out_slot,
                                                    int32_t* __restrict__ inst_fill)
{
    constexpr int NT = NTB, NWAVE = NTB / 64;
    __shared__ int used[2][APC_MAX_LEVELS + 1];
    __shared__ int wcnt[NWAVE][APC_MAX_LEVELS + 2];          // [L + 1]: the wave has an applicant
    __shared__ AssignTable t;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    float best[QPT];
#pragma unroll
    for (int c = 0; c < QPT; ++c) {                          // issued before the table copy
        const int q = c * NT + tid;
        best[c] = q < b ? top_score[(int64_t)q * ld] : 0.f;
    }
    table_to_lds<NT>(targ, t, tid);
    const int L = t.L;
    const uint64_t lt_mask = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
    int lam[QPT], lev[QPT], rk[QPT];
#pragma unroll
    for (int c = 0; c < QPT; ++c) {
        const int q = c * NT + tid;
        lam[c] = 0;
        lev[c] = -1;
        rk[c] = -1;
        if (q < b)
            for (int l = 0; l < L; ++l) lam[c] += best[c] >= t.theta[l];
    }
    if (tid <= L) used[0][tid] = 0;
    int cur = 0;
    const int nchunk = (b + NT - 1) / NT;
    for (int r = 0; r <= L; ++r) {
        bool round_any = false;
#pragma unroll
        for (int c = 0; c < QPT; ++c) {
            if (c < nchunk) {                                 // uniform
                const int q = c * NT + tid;
                int want = -1;
                if (q < b && lev[c] < 0) want = r <= lam[c] ? lam[c] - r : r;
                int pre = 0;
                for (int p = 0; p <= L; ++p) {
                    const uint64_t m = __ballot(want == p);
                    if (want == p) pre = __popcll(m & lt_mask);
                    if (lane == 0) wcnt[wave][p] = __popcll(m);
                }
                const bool wave_any = __ballot(want >= 0) != 0;
                if (lane == 0) wcnt[wave][L + 1] = wave_any;
                __syncthreads();
                bool any = false;
#pragma unroll
                for (int w = 0; w < NWAVE; ++w) any |= wcnt[w][L + 1] != 0;
                if (!any) {                                   // uniform: no applicant in this chunk
                    __syncthreads();                          // before the next chunk rewrites wcnt
                    continue;
                }
                round_any = true;
                if (want >= 0) {
                    int rank = used[cur][want] + pre;
#pragma unroll
                    for (int w = 0; w < NWAVE; ++w) rank += w < wave ? wcnt[w][want] : 0;
                    if (rank < t.level_cap[want]) {
                        lev[c] = want;
                        rk[c] = rank;
                    }
                }
                if (tid <= L) {
                    int tot = used[cur][tid];
#pragma unroll
                    for (int w = 0; w < NWAVE; ++w) tot += wcnt[w][tid];
                    const int cap = t.level_cap[tid];
                    used[cur ^ 1][tid] = tot < cap ? tot : cap;
                }
                __syncthreads();
                cur ^= 1;
            }
        }
        if (!round_any) break;                                // uniform
    }
#pragma unroll
    for (int c = 0; c < QPT; ++c) {
        const int q = c * NT + tid;
        if (q >= b) continue;
        const int p = lev[c];
        int inst = -1, slot = -1;
        if (p >= 0) {
            for (int j = t.level_first[p]; j < t.level_first[p + 1]; ++j)
                if (rk[c] < t.ord_cum[j] + t.ord_cap[j]) {
                    inst = t.ord_inst[j];
                    slot = rk[c] - t.ord_cum[j];
                    break;
                }
        }
        opt_level[q] = lam[c];
        out_level[q] = p;
        out_inst[q] = inst;
        out_slot[q] = slot;
    }
    for (int p = 0; p <= L; ++p)
        for (int j = t.level_first[p] + tid; j < t.level_first[p + 1]; j += NT) {
            int f = used[cur][p] - t.ord_cum[j];
            f = f < 0 ? 0 : (f > t.ord_cap[j] ? t.ord_cap[j] : f);
            inst_fill[t.ord_inst[j]] = f;
        }
}

// Position of level j in the preference list of level i, and its inverse.
__device__ inline int pref_pos(int i, int j) { return j == i ? 0 : (j < i ? i - j : j); }
__device__ inline int pref_at(int i, int pos) { return pos == 0 ? i : (pos <= i ? i - pos : pos); }

// Placement that follows a route plan x (queries of optimal level i served
// at level j).  Same block shape and per-thread query ownership as
// k_assign_reg.  Pass 1 ranks every query among the queries of its own level
// in index order (per-level ballots, per-wave totals, chunks in order), which
// also yields the batch's level histogram H.  With PLANNED the block then
// builds the optimal plan from H, the places per level and K (one thread per
// level, then one per plan entry) and writes it out; otherwise it reads the
// caller's plan (negative entries count as 0).  A query of level i with rank
// s takes the first level j of its preference list [i, i-1, .., 0, i+1, .., L]
// where s falls below the running sum of x[i][.]; the position pos of j in
// that list is its round.  A level admits in (round, index) order while it
// has places, so a query's admission rank is the number of queries routed to
// j in earlier rounds (from the realised flow) plus its rank inside group
// (j, pos).  Only group (j, j) mixes queries of several levels; pass 2 ranks
// its members with one ballot per such level, the others are ranked by their
// offset in their level's quota.
template <int QPT, int NTB, bool PLANNED>
__global__ __launch_bounds__(NTB) void k_assign_plan(const AssignTable targ, const float* __restrict__ top_score,
                                                     int32_t ld, int32_t b, int32_t* __restrict__ plan,
                                                     int32_t* __restrict__ opt_level,
                                                     int32_t* __restrict__ out_level,
                                                     int32_t* __restrict__ out_inst,
                                                     int32_t* __restrict__ out_slot,
                                                     int32_t* __restrict__ inst_fill)
{
    constexpr int NT = NTB, NWAVE = NTB / 64, NL = APC_MAX_LEVELS + 1;
    __shared__ int cnt[2][NL];
    __shared__ int wcnt[NWAVE][NL];
    __shared__ int xs[NL * NL];
    __shared__ int fs[NL * NL];                              // realised flow, level i -> level j
    __shared__ int gb[NL * NL];                              // [j * n + pos]: places before group (j, pos)
    __shared__ int used[NL];                                 // places taken per level
    __shared__ int cnt2[2][NL];
    __shared__ PlanWork w;
    __shared__ unsigned long long multi;                     // bit j: group (j, j) has members
    __shared__ AssignTable t;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    float best[QPT];
#pragma unroll
    for (int c = 0; c < QPT; ++c) {
        const int q = c * NT + tid;
        best[c] = q < b ? top_score[(int64_t)q * ld] : 0.f;
    }
    table_to_lds<NT>(targ, t, tid);
    const int L = t.L, n = L + 1;
    const uint64_t lt_mask = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
    const int nchunk = (b + NT - 1) / NT;
    int lam[QPT], rs[QPT], dr[QPT], ik[QPT], rk[QPT];
#pragma unroll
    for (int c = 0; c < QPT; ++c) {
        const int q = c * NT + tid;
        lam[c] = -1;
        rk[c] = -1;
        if (q < b) {
            lam[c] = 0;
            for (int l = 0; l < L; ++l) lam[c] += best[c] >= t.theta[l];
        }
    }
    if (tid <= L) cnt[0][tid] = 0;
    int cur = 0;
    // Pass 1: rank among the queries of the same level; the histogram.
#pragma unroll
    for (int c = 0; c < QPT; ++c) {
        if (c < nchunk) {                                     // uniform
            int pre = 0;
            for (int p = 0; p <= L; ++p) {
                const uint64_t m = __ballot(lam[c] == p);
                if (lam[c] == p) pre = __popcll(m & lt_mask);
                if (lane == 0) wcnt[wave][p] = __popcll(m);
            }
            __syncthreads();
            if (lam[c] >= 0) {
                int r = cnt[cur][lam[c]] + pre;
#pragma unroll
                for (int ww = 0; ww < NWAVE; ++ww) r += ww < wave ? wcnt[ww][lam[c]] : 0;
                rs[c] = r;
            }
            if (tid <= L) {
                int tot = cnt[cur][tid];
#pragma unroll
                for (int ww = 0; ww < NWAVE; ++ww) tot += wcnt[ww][tid];
                cnt[cur ^ 1][tid] = tot;
            }
            __syncthreads();
            cur ^= 1;
        }
    }
    __syncthreads();                                          // b = 0: cnt[0] initialised
    // The plan.
    if (PLANNED) {
        if (tid <= L) plan_level_own(L, cnt[cur], t.level_cap, tid, w);
        __syncthreads();
        if (tid < L) plan_level_flow(L, tid, w);
        if (tid == L) w.n[L] = 0;
        __syncthreads();
        if (tid <= L) plan_level_intervals(L, tid, w);
        __syncthreads();
        for (int e = tid; e < n * n; e += NT) {
            const int v = plan_entry(e / n, e % n, w);
            xs[e] = v;
            plan[e] = v;
        }
    } else {
        for (int e = tid; e < n * n; e += NT) {
            const int v = plan[e];
            xs[e] = v < 0 ? 0 : v;
        }
    }
    __syncthreads();
    // Realised flow: how many of level i's queries the plan sends to level j
    // (the row's quotas taken in preference order until the level runs out).
    const int* H = cnt[cur];
    for (int e = tid; e < n * n; e += NT) {
        const int i = e / n, j = e - i * n, pj = pref_pos(i, j);
        int64_t before = 0;
        for (int pos = 0; pos < pj; ++pos) before += xs[i * n + pref_at(i, pos)];
        int64_t f = (int64_t)H[i] - before;
        f = f < 0 ? 0 : (f > xs[e] ? xs[e] : f);
        fs[e] = (int)f;
    }
    if (tid == 0) multi = 0ull;
    __syncthreads();
    // Places at level j taken before group (j, pos), i.e. by earlier positions.
    for (int e = tid; e < n * n; e += NT) {
        const int j = e / n, pos = e - j * n;
        int base = 0;
        for (int i = 0; i <= L; ++i) base += pref_pos(i, j) < pos ? fs[i * n + j] : 0;
        gb[e] = base;
    }
    if (tid <= L) {
        int tot = 0;
        for (int i = 0; i <= L; ++i) tot += fs[i * n + tid];
        used[tid] = tot < t.level_cap[tid] ? tot : t.level_cap[tid];
        cnt2[0][tid] = 0;
    }
    // Destination, position and rank inside its group (j, pos).  A group with
    // pos != j holds queries of one level i only (i = j + pos, or i = j for
    // pos = 0), in index order, so the rank is the offset in i's quota.  Group
    // (j, j) gathers the moves up from every level below j (and the move down
    // from level 2j): ranked by ballots below.
#pragma unroll
    for (int c = 0; c < QPT; ++c) {
        dr[c] = -1;
        ik[c] = -1;
        if (c < nchunk && lam[c] >= 0) {
            const int i = lam[c];
            int64_t acc = 0;
            for (int pos = 0; pos <= L; ++pos) {
                const int j = pref_at(i, pos);
                const int x = xs[i * n + j];
                acc += x;
                if (rs[c] < acc) {
                    dr[c] = j | (pos << 8);
                    if (pos == j && j > 0) atomicOr(&multi, 1ull << j);
                    else ik[c] = rs[c] - (int)(acc - x);
                    break;
                }
            }
        }
    }
    __syncthreads();
    const unsigned long long mm = multi;
    cur = 0;
    if (mm) {                                                 // uniform
#pragma unroll
        for (int c = 0; c < QPT; ++c) {
            if (c < nchunk) {                                 // uniform
                const int g = (dr[c] >= 0 && ik[c] < 0) ? (dr[c] & 0xff) : -1;
                int pre = 0;
                for (unsigned long long bits = mm; bits; bits &= bits - 1) {
                    const int j = __builtin_ctzll(bits);
                    const uint64_t m = __ballot(g == j);
                    if (g == j) pre = __popcll(m & lt_mask);
                    if (lane == 0) wcnt[wave][j] = __popcll(m);
                }
                __syncthreads();
                if (g >= 0) {
                    int r = cnt2[cur][g] + pre;
#pragma unroll
                    for (int ww = 0; ww < NWAVE; ++ww) r += ww < wave ? wcnt[ww][g] : 0;
                    ik[c] = r;
                }
                if (tid <= L && ((mm >> tid) & 1ull)) {
                    int tot = cnt2[cur][tid];
#pragma unroll
                    for (int ww = 0; ww < NWAVE; ++ww) tot += wcnt[ww][tid];
                    cnt2[cur ^ 1][tid] = tot;
                }
                __syncthreads();
                cur ^= 1;
            }
        }
    }
    // Admission rank at the level: earlier groups, then the rank in the group.
#pragma unroll
    for (int c = 0; c < QPT; ++c) {
        rk[c] = -1;
        if (dr[c] >= 0) {
            const int j = dr[c] & 0xff, pos = dr[c] >> 8;
            const int rank = gb[j * n + pos] + ik[c];
            if (rank < t.level_cap[j]) rk[c] = rank;
        }
    }
#pragma unroll
    for (int c = 0; c < QPT; ++c) {
        const int q = c * NT + tid;
        if (q >= b) continue;
        const int p = rk[c] >= 0 ? (dr[c] & 0xff) : -1;
        int inst = -1, slot = -1;
        if (p >= 0) {
            for (int j = t.level_first[p]; j < t.level_first[p + 1]; ++j)
                if (rk[c] < t.ord_cum[j] + t.ord_cap[j]) {
                    inst = t.ord_inst[j];
                    slot = rk[c] - t.ord_cum[j];
                    break;
                }
        }
        opt_level[q] = lam[c];
        out_level[q] = p;
        out_inst[q] = inst;
        out_slot[q] = slot;
    }
    for (int p = 0; p <= L; ++p)
        for (int j = t.level_first[p] + tid; j < t.level_first[p + 1]; j += NT) {
            int f = used[p] - t.ord_cum[j];
            f = f < 0 ? 0 : (f > t.ord_cap[j] ? t.ord_cap[j] : f);
            inst_fill[t.ord_inst[j]] = f;
        }
}

template <bool PLANNED>
hipError_t launch_plan_t(const AssignTable& t, const float* top_score, int32_t ld, int32_t b, int32_t* plan,
                         int32_t* opt_level, int32_t* out_level, int32_t* out_inst, int32_t* out_slot,
                         int32_t* inst_fill, hipStream_t s)
{
    if (b <= 256)
        k_assign_plan<1, 256, PLANNED><<<1, 256, 0, s>>>(t, top_score, ld, b, plan, opt_level, out_level, out_inst, out_slot, inst_fill);
    else if (b <= NT)
        k_assign_plan<1, NT, PLANNED><<<1, NT, 0, s>>>(t, top_score, ld, b, plan, opt_level, out_level, out_inst, out_slot, inst_fill);
    else if (b <= 4 * NT)
        k_assign_plan<4, NT, PLANNED><<<1, NT, 0, s>>>(t, top_score, ld, b, plan, opt_level, out_level, out_inst, out_slot, inst_fill);
    else if (b <= 16 * NT)
        k_assign_plan<16, NT, PLANNED><<<1, NT, 0, s>>>(t, top_score, ld, b, plan, opt_level, out_level, out_inst, out_slot, inst_fill);
    else
        return hipErrorInvalidValue;
    return hipGetLastError();
}

}  // namespace

hipError_t launch_assign(const AssignTable& t, const float* top_score, int32_t ld, int32_t b,
                         int32_t* opt_level, int32_t* out_level, int32_t* out_inst,
                         int32_t* out_slot, int32_t* inst_fill, hipStream_t s)
{
    if (b <= 256)
        k_assign_reg<1, 256><<<1, 256, 0, s>>>(t, top_score, ld, b, opt_level, out_level, out_inst, out_slot, inst_fill);
    else if (b <= NT)
        k_assign_reg<1, NT><<<1, NT, 0, s>>>(t, top_score, ld, b, opt_level, out_level, out_inst, out_slot, inst_fill);
    else if (b <= 4 * NT)
        k_assign_reg<4, NT><<<1, NT, 0, s>>>(t, top_score, ld, b, opt_level, out_level, out_inst, out_slot, inst_fill);
    else if (b <= 16 * NT)
        k_assign_reg<16, NT><<<1, NT, 0, s>>>(t, top_score, ld, b, opt_level, out_level, out_inst, out_slot, inst_fill);
    else
        k_assign<<<1, NT, 0, s>>>(t, top_score, ld, b, opt_level, out_level, out_inst, out_slot, inst_fill);
    return hipGetLastError();
}

hipError_t launch_assign_plan(const AssignTable& t, bool planned, const float* top_score, int32_t ld, int32_t b,
                              int32_t* plan, int32_t* opt_level, int32_t* out_level, int32_t* out_inst,
                              int32_t* out_slot, int32_t* inst_fill, hipStream_t s)
{
    static_assert(16 * NT == APC_MAX_ROUTED_BATCH, "largest routed batch");
    return planned ? launch_plan_t<true>(t, top_score, ld, b, plan, opt_level, out_level, out_inst, out_slot, inst_fill, s)
                   : launch_plan_t<false>(t, top_score, ld, b, plan, opt_level, out_level, out_inst, out_slot, inst_fill, s);
}

}  // namespace apc
