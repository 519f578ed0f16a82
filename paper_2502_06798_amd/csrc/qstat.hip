// Query-stationary similarity + top-k for small batches (the HBM-bound regime).
//
// Each wavefront keeps its MQ x 32 queries resident in VGPRs for its whole
// life (as MFMA B operands), so one workgroup of four wavefronts covers
// 4 x MQ x 32 queries and every cache row is read from HBM once per
// workgroup.  Cache rows stream through LDS in stages of 32 rows x 256 bytes
// with direct-to-LDS loads (no registers held by loads in flight; twelve
// stages = 96 KB in flight per CU).  Each lane fetches the 16-byte unit
// that lands where an XOR swizzle wants it, so the MFMA A-operand reads
// (lane = row, 16 bytes per step) are free of bank conflicts.  One barrier
// per stage makes the stage visible to all four wavefronts.  The entry
// factors of a 32-row block come in through the same pipeline (one more
// direct load with the block's first stage) into a small LDS ring.
//
// Lane l supplies row l % 32 of a 32x32 block; half h = l / 32 supplies the
// bytes [64h, 64h + 64) of every 128-byte chunk of d, for cache rows (from
// LDS) and query rows (from VGPRs) alike.  In the 32x32 result, lane (h, c)
// holds column (query) c for the 16 rows 8g + 4h + i (g, i < 4).
//
// Top-k: both lanes of a query keep a sorted list of the best pairs among
// their own rows, in registers.  A lane admits a pair only if it comes before
// the admission threshold: the later of its own k-th pair and its partner
// lane's k-th pair.  Either is a pair with k pairs at or before it, so a pair
// that does not come before it is not in the top-k of the rows seen, and the
// pair itself is already kept by the lane that owns it.  At the end the
// partner's list is merged into lane h = 0, which writes the split's list.
#include <type_traits>

#include "topk_wg.h"

namespace apc {
namespace {

typedef __attribute__((address_space(3))) void lds_void;

constexpr int QS_NW = 4;              // wavefronts per workgroup
constexpr int QS_NT = QS_NW * 64;
constexpr int QS_SB = 256;            // bytes of every row per stage
constexpr int QS_STAGE = 32 * QS_SB;  // 8 KB: 32 rows
constexpr int QS_NS = 12;             // stages in LDS
constexpr int QS_LPW = QS_STAGE / 1024 / QS_NW;   // row loads per wavefront per stage
constexpr int QS_FR = 16;             // entry-factor ring: blocks
constexpr int QS_KR = 16;             // largest k

// s_waitcnt immediate that waits until at most n vector-memory operations are
// outstanding (and does not wait on the other counters)
constexpr int vmcnt_imm(int n) { return (n & 15) | (((n >> 4) & 3) << 14) | (7 << 4) | (15 << 8); }

// 16 bytes per lane from global memory straight into LDS: lane l's bytes land
// at lds + 16 l.  Written as an asm statement so that the compiler does not
// treat every later LDS read as dependent on all loads in flight (it would
// wait for the whole pipeline before each read); the kernel waits on the
// vector-memory counter itself.
__device__ inline void dma16(const void* g, uint32_t lds)
{
    asm volatile("s_nop 0\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(g), "{m0}"(lds) : "memory");
}

// A step is what one lane feeds one MFMA: 16 bytes (8 halves), or for e4m3
// 32 bytes (two 16-byte units, 32 codes).
template <int DT> struct QsStep { typedef uint4 type; static constexpr int UNITS = 1; };
template <> struct QsStep<APC_E4M3> { typedef i32x8 type; static constexpr int UNITS = 2; };

template <int DT, int RB, int MQ>
struct QsCfg {
    typedef typename QsStep<DT>::type Step;
    static constexpr int UPS = QsStep<DT>::UNITS;     // 16-byte units per step
    static constexpr int QU = RB / 32;                // 16-byte units of a query row held by a lane
    static constexpr int QST = QU / UPS;              // steps of a query row held by a lane
    static constexpr int SST = QS_SB / 32 / UPS;      // steps per stage
    static constexpr int SPB = RB / QS_SB;            // stages per 32-row block
    static constexpr int BQW = MQ * 32;               // queries per wavefront
    static constexpr int BQ = QS_NW * BQW;            // queries per workgroup
    static_assert(RB % QS_SB == 0, "rows must be whole stages");
    static_assert(SPB >= 2, "the factor ring assumes at least two stages per block");
    static_assert(DT != APC_F32, "float rows use the streaming kernel");
    // vector-memory operations a wavefront issues after stage t (static j = t % SPB)
    // and before stage t's wait, in steady state: stages t+1 .. t+NS-2, plus one
    // factor load for each block start among them
    static constexpr int after(int j) { return (QS_NS - 2) * QS_LPW + (j + QS_NS - 2) / SPB; }
    // wait for stage t (j = t % SPB; a constant once the stage loop is unrolled)
    __device__ static void wait_stage(int j)
    {
        static_assert(SPB <= 6, "wait_stage covers up to six stages per block");
        switch (j) {
        case 0: __builtin_amdgcn_s_waitcnt(vmcnt_imm(after(0))); break;
        case 1: __builtin_amdgcn_s_waitcnt(vmcnt_imm(after(1))); break;
        case 2: __builtin_amdgcn_s_waitcnt(vmcnt_imm(after(2))); break;
        case 3: __builtin_amdgcn_s_waitcnt(vmcnt_imm(after(3))); break;
        case 4: __builtin_amdgcn_s_waitcnt(vmcnt_imm(after(4))); break;
        default: __builtin_amdgcn_s_waitcnt(vmcnt_imm(after(5))); break;
        }
    }
    struct Smem {
        uint8_t e[QS_NS * QS_STAGE];
        float fe[QS_FR][32];
    };
};

template <int DT>
__device__ inline void mma_step(f32x16& c, const typename QsStep<DT>::type a, const typename QsStep<DT>::type b)
{
    if constexpr (DT == APC_F16)
        c = __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(f16x8, a), __builtin_bit_cast(f16x8, b), c, 0, 0, 0);
    else if constexpr (DT == APC_BF16)
        c = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
    else
        c = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, b, c, 0, 0, 0, 0, 0, 0);
}

template <int DT>
__device__ inline void sumsq_step(const typename QsStep<DT>::type v, float& ss, bool& bad)
{
    if constexpr (DT == APC_E4M3) {
        sumsq16<DT>(make_uint4(v[0], v[1], v[2], v[3]), ss, bad);
        sumsq16<DT>(make_uint4(v[4], v[5], v[6], v[7]), ss, bad);
    } else {
        sumsq16<DT>(v, ss, bad);
    }
}

// Insert (s, e) into the sorted list (ls, li) of QS_KR pairs, dropping the last.
// Branch-free: position p takes the pair above it if the new pair comes before
// that one, else the new pair if it comes before p's own, else keeps its own.
// (-inf, IDX_NONE) comes before nothing and leaves the list as it is.
__device__ inline void list_insert(float (&ls)[QS_KR], int (&li)[QS_KR], float s, int e)
{
    bool c[QS_KR];
#pragma unroll
    for (int p = 0; p < QS_KR; ++p) c[p] = before(s, e, ls[p], li[p]);
#pragma unroll
    for (int p = QS_KR - 1; p >= 1; --p) {
        ls[p] = c[p - 1] ? ls[p - 1] : (c[p] ? s : ls[p]);
        li[p] = c[p - 1] ? li[p - 1] : (c[p] ? e : li[p]);
    }
    ls[0] = c[0] ? s : ls[0];
    li[0] = c[0] ? e : li[0];
}

// the k-th pair of a list (k is a runtime value <= QS_KR)
__device__ inline void list_kth(const float (&ls)[QS_KR], const int (&li)[QS_KR], int k, float& ts, int& ti)
{
    ts = ls[0];
    ti = li[0];
#pragma unroll
    for (int p = 1; p < QS_KR; ++p) {
        ts = p == k - 1 ? ls[p] : ts;
        ti = p == k - 1 ? li[p] : ti;
    }
}

// Merge the partner lane's sorted list (lane l ^ 32) into this lane's: the
// better of own[p] and partner[KR-1-p] at every p gives the KR best of both
// lists as a bitonic sequence, which four half-cleaner stages sort.
__device__ inline void list_merge_partner(float (&ls)[QS_KR], int (&li)[QS_KR])
{
#pragma unroll
    for (int p = 0; p < QS_KR; ++p) {
        const float bs = __shfl_xor(ls[QS_KR - 1 - p], 32, 64);
        const int bi = __shfl_xor(li[QS_KR - 1 - p], 32, 64);
        const bool take = before(bs, bi, ls[p], li[p]);
        ls[p] = take ? bs : ls[p];
        li[p] = take ? bi : li[p];
    }
#pragma unroll
    for (int st = QS_KR / 2; st >= 1; st /= 2)
#pragma unroll
        for (int p = 0; p < QS_KR; ++p)
            if ((p & st) == 0) {
                const bool sw = before(ls[p + st], li[p + st], ls[p], li[p]);
                const float s0 = ls[p], s1 = ls[p + st];
                const int i0 = li[p], i1 = li[p + st];
                ls[p] = sw ? s1 : s0;
                li[p] = sw ? i1 : i0;
                ls[p + st] = sw ? s0 : s1;
                li[p + st] = sw ? i0 : i1;
            }
}

// grid: splits * qtiles workgroups.  When splits is a multiple of 8, the
// query tiles of one split get ids 8 apart, so they run on the same XCD
// (workgroups go round-robin over the 8 XCDs) at about the same time and a
// cache row read by one of them is an L2 hit for the others.
template <int DT, int RB, int MQ>
__global__ __launch_bounds__(QS_NT) void k_qstat(
    const uint8_t* __restrict__ emb, const float* __restrict__ fe, int64_t n,
    const uint8_t* __restrict__ qry, const float* __restrict__ q_scale, int32_t b, int32_t k,
    int splits, int qtiles, int64_t b_pad, float* __restrict__ fq_out, float* __restrict__ part_s,
    int* __restrict__ part_i)
{
    typedef QsCfg<DT, RB, MQ> C;
    typedef typename C::Step Step;
    __shared__ typename C::Smem sm;
    const int tid = threadIdx.x, lane = tid & 63, h = lane >> 5, r32 = lane & 31;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    int split, qtile;
    if ((splits & 7) == 0) {
        const int rest = blockIdx.x >> 3;
        qtile = rest % qtiles;
        split = (rest / qtiles) * 8 + (blockIdx.x & 7);
    } else {
        split = blockIdx.x % splits;
        qtile = blockIdx.x / splits;
    }
    const int64_t q0 = (int64_t)qtile * C::BQ + wave * C::BQW;   // this wavefront's first query
    const bool live = q0 < b;                                      // uniform per wavefront

    const int64_t nblk = (n + 31) / 32;
    const int64_t b_begin = nblk * split / splits;
    const int nb = (int)(nblk * (split + 1) / splits - b_begin);  // blocks of this workgroup
    const int T = nb * C::SPB;                                     // stages of this workgroup

    // ---- stage loads: wavefront w fills rows [8w, 8w + 8) of a stage ----
    // lane l of load i writes LDS unit (l % 16) of row 8w + 4i + l / 16; that unit
    // holds logical unit (l % 16) ^ (row % 16) of the row's stage bytes
    const uint32_t lds_e = (uint32_t)(size_t)(lds_void*)sm.e;
    const uint32_t lds_f = (uint32_t)(size_t)(lds_void*)&sm.fe[0][0];
    int lrow[QS_LPW], loff[QS_LPW];
#pragma unroll
    for (int i = 0; i < QS_LPW; ++i) {
        lrow[i] = wave * (32 / QS_NW) + i * 4 + (lane >> 4);
        loff[i] = ((lane & 15) ^ (lrow[i] & 15)) * 16;
    }
    auto issue_stage = [&](int t) {
        const int bl = t / C::SPB, j = t - bl * C::SPB;
        const int64_t blk = b_begin + bl;
        const int64_t last = n - 1 - blk * 32;                     // last valid row in the block
        const uint8_t* gb = emb + blk * 32 * RB + j * QS_SB;
        const uint32_t sbase = lds_e + (uint32_t)(t % QS_NS) * QS_STAGE;
#pragma unroll
        for (int i = 0; i < QS_LPW; ++i) {
            const int row = lrow[i] < last ? lrow[i] : (int)last;
            dma16(gb + row * RB + loff[i], __builtin_amdgcn_readfirstlane(sbase + (wave * (32 / QS_NW) + i * 4) * QS_SB));
        }
        if (j == 0 && lane < 8)       // the block's 32 entry factors (fe is padded to whole blocks)
            dma16(fe + blk * 32 + lane * 4, lds_f + (uint32_t)(bl % QS_FR) * 128);
    };
#pragma unroll
    for (int s = 0; s < QS_NS - 1; ++s)
        if (s < T) issue_stage(s);

    // ---- queries into VGPRs; their factors ----
    // lane (h, r32) holds, of query row mq * 32 + r32, the bytes [64h, 64h + 64)
    // of every 128-byte chunk; step s covers units UPS*s .. UPS*s + UPS - 1
    Step qv[C::QST][MQ];
    float fqv[MQ];
    // one query row per call, with a compile-time row index so that qv stays
    // in registers (a loop over the rows may be left rolled: its body is large)
    auto prep = [&](auto mqc) __attribute__((always_inline)) {
        constexpr int mq = decltype(mqc)::value;
        const int64_t qg = q0 + mq * 32 + r32;
        const bool ok_row = qg < b;
        const uint8_t* qrow = qry + (ok_row ? qg : 0) * RB + h * 64;
#pragma unroll
        for (int s = 0; s < C::QST; ++s) {
            const int u = s * C::UPS;
            qv[s][mq] = *reinterpret_cast<const Step*>(qrow + (u / 4) * 128 + (u % 4) * 16);
        }
        float ss = 0.f;
        bool bad = false;
#pragma unroll
        for (int s = 0; s < C::QST; ++s) sumsq_step<DT>(qv[s][mq], ss, bad);
        ss += __shfl_xor(ss, 32, 64);
        bad = bad || __shfl_xor((int)bad, 32, 64);
        bool ok = ok_row && !bad && __builtin_isfinite(ss) && ss > 0.f;
        if (ok && q_scale) {
            const float sc = q_scale[qg];
            ok = __builtin_isfinite(sc) && sc > 0.f;
        }
        fqv[mq] = ok ? 1.0f / __builtin_sqrtf(ss) : qnan();
        if (split == 0 && h == 0 && ok_row) fq_out[qg] = fqv[mq];
    };
    prep(std::integral_constant<int, 0>{});
    if constexpr (MQ > 1) prep(std::integral_constant<int, 1>{});
    static_assert(MQ <= 2, "one or two query blocks per wavefront");

    // ---- per-lane lists and admission thresholds ----
    float ls[MQ][QS_KR];
    int li[MQ][QS_KR];
    float ts[MQ];      // admission threshold: the later of own and partner's k-th pair
    int ti[MQ];
#pragma unroll
    for (int mq = 0; mq < MQ; ++mq) {
#pragma unroll
        for (int p = 0; p < QS_KR; ++p) {
            ls[mq][p] = neg_inf();
            li[mq][p] = IDX_NONE;
        }
        ts[mq] = neg_inf();
        ti[mq] = IDX_NONE;
    }

    f32x16 acc[MQ];
#pragma unroll
    for (int mq = 0; mq < MQ; ++mq)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[mq][r] = 0.f;

    for (int bi = 0; bi < nb; ++bi) {
#pragma unroll
        for (int j = 0; j < C::SPB; ++j) {                        // stage j of the block: static, so
            const int t = bi * C::SPB + j;                        // the query steps index registers
            // stage t is in when at most (loads issued after it) are outstanding
            if (t + QS_NS - 2 < T) C::wait_stage(j);
            else __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));
            __syncthreads();
            if (t + QS_NS - 1 < T) issue_stage(t + QS_NS - 1);   // into the slot stage t - 1 used
            if (!live) continue;

            const uint8_t* srow = sm.e + (t % QS_NS) * QS_STAGE + r32 * QS_SB;
            // all LDS reads of the stage first, then the MFMAs
            Step a[C::SST];
#pragma unroll
            for (int ss = 0; ss < C::SST; ++ss) {
                const int cl = ss / (4 / C::UPS), sp = ss % (4 / C::UPS);
                const int lu = cl * 8 + h * 4 + sp * C::UPS;              // logical unit in the stage
                if constexpr (C::UPS == 1) {
                    a[ss] = *reinterpret_cast<const uint4*>(srow + ((lu ^ (r32 & 15)) * 16));
                } else {
                    const uint4 x0 = *reinterpret_cast<const uint4*>(srow + ((lu ^ (r32 & 15)) * 16));
                    const uint4 x1 = *reinterpret_cast<const uint4*>(srow + (((lu + 1) ^ (r32 & 15)) * 16));
                    a[ss] = i32x8{(int)x0.x, (int)x0.y, (int)x0.z, (int)x0.w,
                                  (int)x1.x, (int)x1.y, (int)x1.z, (int)x1.w};
                }
            }
#pragma unroll
            for (int ss = 0; ss < C::SST; ++ss)
#pragma unroll
                for (int mq = 0; mq < MQ; ++mq) mma_step<DT>(acc[mq], a[ss], qv[j * C::SST + ss][mq]);
            // keep the reads ahead of the MFMAs (the scheduler would otherwise
            // pair each read with its MFMA and wait out every read's latency)
            __builtin_amdgcn_sched_group_barrier(0x100, C::SST * C::UPS, 0);
            __builtin_amdgcn_sched_group_barrier(0x008, C::SST * MQ, 0);
        }
        if (!live) continue;

        // ---- epilogue of the block: scores, admission, insertion ----
        const int64_t blk = b_begin + bi;
        const int lim = (int)(n - blk * 32 - 4 * h < 64 ? n - blk * 32 - 4 * h : 64);
        const int ebase = (int)(blk * 32) + 4 * h;
        float fev[16];
        {
            const float* fr = sm.fe[bi % QS_FR];
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                const float4 v = *reinterpret_cast<const float4*>(fr + 8 * g + 4 * h);
                fev[4 * g + 0] = v.x;
                fev[4 * g + 1] = v.y;
                fev[4 * g + 2] = v.z;
                fev[4 * g + 3] = v.w;
            }
        }
        uint32_t pend[MQ];
        bool any_pend = false;
#pragma unroll
        for (int mq = 0; mq < MQ; ++mq) {
            float m = neg_inf();
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const float v = acc[mq][r] * fev[r];
                acc[mq][r] = v;
                if (8 * (r >> 2) + (r & 3) < lim) m = __builtin_fmaxf(m, v);
            }
            const float f = fqv[mq];
            const float mx = (m == neg_inf() || !(f == f)) ? neg_inf() : clamp1(m * f);
            pend[mq] = 0;
            if (mx >= ts[mq] && mx > neg_inf()) {
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const float sc = clamp1(acc[mq][r] * f);
                    acc[mq][r] = sc;
                    const int e = ebase + 8 * (r >> 2) + (r & 3);
                    if (8 * (r >> 2) + (r & 3) < lim && before(sc, e, ts[mq], ti[mq])) pend[mq] |= 1u << r;
                }
            }
            any_pend |= pend[mq] != 0;
        }
        if (__any(any_pend)) {
#pragma unroll
            for (int mq = 0; mq < MQ; ++mq) {
                // one admitted pair per lane and pass, lowest row first; lanes with
                // nothing left insert (-inf, IDX_NONE), which changes nothing, so
                // the pass has no branches (and the list stays in place)
                while (__any(pend[mq] != 0)) {
                    const bool has = pend[mq] != 0;
                    const int r = __builtin_ctz(pend[mq] | 0x10000u);
                    pend[mq] &= pend[mq] - 1;
                    float sc = acc[mq][0];
#pragma unroll
                    for (int rr = 1; rr < 16; ++rr) sc = r == rr ? acc[mq][rr] : sc;
                    int e = ebase + 8 * (r >> 2) + (r & 3);
                    const bool ok = has && before(sc, e, ts[mq], ti[mq]);
                    sc = ok ? sc : neg_inf();
                    e = ok ? e : IDX_NONE;
                    list_insert(ls[mq], li[mq], sc, e);
                    float own_s;
                    int own_i;
                    list_kth(ls[mq], li[mq], k, own_s, own_i);
                    const bool up = before(own_s, own_i, ts[mq], ti[mq]);
                    ts[mq] = up ? own_s : ts[mq];
                    ti[mq] = up ? own_i : ti[mq];
                }
                // the partner lane's k-th pair may now be the later one
                float own_s;
                int own_i;
                list_kth(ls[mq], li[mq], k, own_s, own_i);
                const float partner_s = __shfl_xor(own_s, 32, 64);
                const int partner_i = __shfl_xor(own_i, 32, 64);
                const bool up = before(partner_s, partner_i, ts[mq], ti[mq]);
                ts[mq] = up ? partner_s : ts[mq];
                ti[mq] = up ? partner_i : ti[mq];
            }
        }
#pragma unroll
        for (int mq = 0; mq < MQ; ++mq)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[mq][r] = 0.f;
    }

    if (!live) return;
    // ---- merge the partner's list into lane h = 0 and write the split's lists ----
#pragma unroll
    for (int mq = 0; mq < MQ; ++mq) {
        list_merge_partner(ls[mq], li[mq]);
        const int64_t qg = q0 + mq * 32 + r32;
        if (h == 0 && qg < b_pad) {
            const int64_t o = ((int64_t)qg * splits + split) * k;
#pragma unroll
            for (int p = 0; p < QS_KR; ++p)
                if (p < k) {
                    part_s[o + p] = ls[mq][p];
                    part_i[o + p] = li[mq][p];
                }
        }
    }
}

template <int DT, int RB, int MQ>
hipError_t run_qstat(const MatchPlan& p, int64_t n, const void* emb, const float* fe, const void* q,
                     const float* q_scale, int32_t b, int32_t k, float* fq, float* ps, int* pi,
                     hipStream_t s)
{
    const dim3 grid((unsigned)(p.splits * p.qtiles)), block(QS_NT);
    k_qstat<DT, RB, MQ><<<grid, block, 0, s>>>(static_cast<const uint8_t*>(emb), fe, n,
                                               static_cast<const uint8_t*>(q), q_scale, b, k, p.splits,
                                               p.qtiles, p.b_pad, fq, ps, pi);
    return hipGetLastError();
}

}  // namespace

// queries per workgroup of the query-stationary kernel for this row size, 0 if not built.
// A lane holds half of each of its MQ query rows in registers: MQ = 2 up to
// 1 KB rows, MQ = 1 for 1.5 KB rows (192 VGPRs of queries).
int qstat_queries(int dt, int64_t row_bytes)
{
    switch (dt) {
    case APC_F16: case APC_BF16:
        return row_bytes == 1536 ? QsCfg<APC_F16, 1536, 1>::BQ
             : row_bytes == 1024 ? QsCfg<APC_F16, 1024, 2>::BQ
             : row_bytes == 512 ? QsCfg<APC_F16, 512, 2>::BQ : 0;
    case APC_E4M3:
        return row_bytes == 768 ? QsCfg<APC_E4M3, 768, 2>::BQ
             : row_bytes == 512 ? QsCfg<APC_E4M3, 512, 2>::BQ : 0;
    default: return 0;
    }
}

hipError_t launch_qstat(const MatchPlan& p, int dt, int64_t n, int32_t d, const void* emb,
                        const float* fe, const void* q, const float* q_scale, int32_t b, int32_t k,
                        float* fq, float* ps, int* pi, hipStream_t s)
{
    const int64_t rb = (int64_t)d * elem_bytes(dt);
#define APC_QS(DT, RB, MQ) run_qstat<DT, RB, MQ>(p, n, emb, fe, q, q_scale, b, k, fq, ps, pi, s)
    switch (dt) {
    case APC_F16:
        return rb == 1536 ? APC_QS(APC_F16, 1536, 1) : rb == 1024 ? APC_QS(APC_F16, 1024, 2) : APC_QS(APC_F16, 512, 2);
    case APC_BF16:
        return rb == 1536 ? APC_QS(APC_BF16, 1536, 1) : rb == 1024 ? APC_QS(APC_BF16, 1024, 2) : APC_QS(APC_BF16, 512, 2);
    case APC_E4M3:
        return rb == 768 ? APC_QS(APC_E4M3, 768, 2) : APC_QS(APC_E4M3, 512, 2);
    default: return hipErrorInvalidValue;
    }
#undef APC_QS
}

}  // namespace apc
