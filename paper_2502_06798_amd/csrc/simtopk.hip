// Nearest cached prompts: cosine similarity of every query against every
// cache entry, fused with an exact per-query top-k.
//
// k_simtopk  - one workgroup owns a tile of BQ queries and a contiguous range
//              of entries (a "split").  It streams entry tiles of BE rows; per
//              tile, MFMA 32x32 blocks accumulate <e, q> over all of d in
//              float32 (entries are the MFMA rows, queries the columns), the
//              operands staged through LDS 128 bytes of each row at a time.
//              The score s = clamp(acc * f_e * f_q, -1, 1) never leaves
//              registers: each lane tests its scores against the per-query
//              threshold (the current k-th best of the workgroup's range, in
//              the order score desc / index asc) and appends the few that
//              pass to small per-query LDS buffers; one thread per query then
//              inserts them into that query's sorted list in LDS.  Buffers
//              that overflow are retried in further rounds after the
//              threshold has risen, so nothing that belongs to the top-k is
//              ever dropped.  At the end the workgroup writes its k best per
//              query (a partial list) to the workspace.
// k_topk_merge - one wavefront per query merges the partial lists of all
//              splits (each sorted, ranges disjoint) by repeated wave argmax.
//
// Every score is produced by the same fixed sequence of MFMAs whatever the
// tiling, and the final list is the unique top-k of those scores under a
// total order, so results are deterministic.
#include "apc_internal.h"

namespace apc {
namespace {

typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef int i32x8 __attribute__((ext_vector_type(8)));

constexpr int KB = 128;          // bytes of each row staged per k-step
constexpr int ROWB = KB + 16;    // LDS row stride: 16 consecutive rows start on distinct bank quads
constexpr int NCAND = 16;        // candidate slots per query per round
constexpr int IDX_NONE = 0x7fffffff;

__device__ inline float neg_inf() { return -__builtin_huge_valf(); }

// (sa, ia) comes before (sb, ib) in the order score desc, index asc
__device__ inline bool before(float sa, int ia, float sb, int ib)
{
    return sa > sb || (sa == sb && ia < ib);
}

// ---- per-type MFMA step over one staged k-step ----------------------------
// Lane l supplies row (l % 32) of its block; lanes l and l + 32 cover the two
// halves of the k-chunk.  A (entries) and B (queries) use the same lane->k
// mapping, which is all the dot product needs.
template <int DT> struct Mma;

template <> struct Mma<APC_F16> {
    static constexpr int NSTEP = 4;                       // 4 x (32x32x16)
    typedef f16x8 Frag;
    __device__ static Frag load(const uint8_t* row, int s, int h)
    {
        return *reinterpret_cast<const Frag*>(row + s * 32 + h * 16);
    }
    __device__ static void mma(f32x16& c, const Frag& a, const Frag& b)
    {
        c = __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, c, 0, 0, 0);
    }
};

template <> struct Mma<APC_BF16> {
    static constexpr int NSTEP = 4;
    typedef bf16x8 Frag;
    __device__ static Frag load(const uint8_t* row, int s, int h)
    {
        return *reinterpret_cast<const Frag*>(row + s * 32 + h * 16);
    }
    __device__ static void mma(f32x16& c, const Frag& a, const Frag& b)
    {
        c = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
    }
};

template <> struct Mma<APC_E4M3> {
    static constexpr int NSTEP = 2;                       // 2 x (32x32x64), OCP e4m3 operands
    typedef i32x8 Frag;
    __device__ static Frag load(const uint8_t* row, int s, int h)
    {
        return *reinterpret_cast<const Frag*>(row + s * 64 + h * 32);
    }
    __device__ static void mma(f32x16& c, const Frag& a, const Frag& b)
    {
        c = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, b, c, 0, 0, 0, 0, 0, 0);
    }
};

template <> struct Mma<APC_F32> {
    static constexpr int NSTEP = 4;                       // 4 x 4 x (32x32x2)
    typedef float4 Frag;
    __device__ static Frag load(const uint8_t* row, int s, int h)
    {
        return *reinterpret_cast<const Frag*>(row + s * 32 + h * 16);
    }
    __device__ static void mma(f32x16& c, const Frag& a, const Frag& b)
    {
        c = __builtin_amdgcn_mfma_f32_32x32x2f32(a.x, b.x, c, 0, 0, 0);
        c = __builtin_amdgcn_mfma_f32_32x32x2f32(a.y, b.y, c, 0, 0, 0);
        c = __builtin_amdgcn_mfma_f32_32x32x2f32(a.z, b.z, c, 0, 0, 0);
        c = __builtin_amdgcn_mfma_f32_32x32x2f32(a.w, b.w, c, 0, 0, 0);
    }
};

// ---- fused similarity + partial top-k ---------------------------------------
// BQ queries x BE entries per tile; WQ x WE wavefronts, each MQ x ME blocks of 32x32.
template <int DT, int BQ, int BE, int WQ, int WE, int KMAX>
struct SimTopk {
    static constexpr int NW = WQ * WE;
    static constexpr int NT = NW * 64;
    static constexpr int MQ = BQ / WQ / 32;
    static constexpr int ME = BE / WE / 32;
    static constexpr int NS = MQ * ME * 16;               // scores per lane per tile
    static constexpr int ROWS = BE + BQ;                  // staged rows (entries first)
    static constexpr int NCH = ROWS * (KB / 16) / NT;     // 16-byte chunks per thread per k-step
    static_assert(NS <= 64, "pending mask holds 64 scores");
    static_assert(ROWS * (KB / 16) % NT == 0, "chunks must divide evenly");
    static_assert(MQ >= 1 && ME >= 1, "tile too small for the wave grid");

    struct Smem {
        uint8_t op[ROWS * ROWB];          // staged operand rows
        float list_s[KMAX * BQ];          // sorted partial top-k, k-major
        int list_i[KMAX * BQ];
        float cand_s[BQ * NCAND];
        int cand_i[BQ * NCAND];
        float thr_s[BQ];                  // k-th best so far (the admission threshold)
        int thr_i[BQ];
        int cnt[BQ];
        float fq[BQ];
    };
};

template <int DT, int BQ, int BE, int WQ, int WE, int KMAX>
__global__ __launch_bounds__(WQ * WE * 64) void k_simtopk(
    const uint8_t* __restrict__ emb, const float* __restrict__ fe, int64_t n,
    const uint8_t* __restrict__ qry, const float* __restrict__ fq, int32_t b,
    int64_t row_bytes, int32_t k, int splits, int64_t b_pad,
    float* __restrict__ part_s, int* __restrict__ part_i)
{
    typedef SimTopk<DT, BQ, BE, WQ, WE, KMAX> P;
    typedef Mma<DT> M;
    __shared__ typename P::Smem sm;

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, h = lane >> 5;
    const int wq = wave / WE, we = wave % WE;
    const int split = blockIdx.x;
    const int64_t q0 = (int64_t)blockIdx.y * BQ;

    const int64_t ntiles = (n + BE - 1) / BE;
    const int64_t t_begin = ntiles * split / splits, t_end = ntiles * (split + 1) / splits;
    const int nks = (int)((row_bytes + KB - 1) / KB);

    // workgroup state: empty lists, thresholds below every score
    for (int i = tid; i < KMAX * BQ; i += P::NT) {
        sm.list_s[i] = neg_inf();
        sm.list_i[i] = IDX_NONE;
    }
    for (int i = tid; i < BQ; i += P::NT) {
        sm.thr_s[i] = neg_inf();
        sm.thr_i[i] = IDX_NONE;
        sm.cnt[i] = 0;
        const int64_t q = q0 + i;
        sm.fq[i] = q < b ? fq[q] : __int_as_float(0x7fc00000);
    }

    uint4 pre[P::NCH];
    auto load_stage = [&](int64_t t, int ks) {
        const int64_t e0 = t * BE;
        const int64_t kb = (int64_t)ks * KB;
#pragma unroll
        for (int j = 0; j < P::NCH; ++j) {
            const int c = tid + j * P::NT;
            const int row = c / (KB / 16), col = c % (KB / 16);
            const int64_t off = kb + col * 16;
            uint4 v = make_uint4(0, 0, 0, 0);
            if (off < row_bytes) {
                if (row < BE) {
                    const int64_t e = e0 + row;
                    if (e < n) v = *reinterpret_cast<const uint4*>(emb + e * row_bytes + off);
                } else {
                    const int64_t q = q0 + (row - BE);
                    if (q < b) v = *reinterpret_cast<const uint4*>(qry + q * row_bytes + off);
                }
            }
            pre[j] = v;
        }
    };

    const uint8_t* a_row[P::ME];
    const uint8_t* b_row[P::MQ];
#pragma unroll
    for (int me = 0; me < P::ME; ++me)
        a_row[me] = sm.op + (we * (BE / WE) + me * 32 + (lane & 31)) * ROWB;
#pragma unroll
    for (int mq = 0; mq < P::MQ; ++mq)
        b_row[mq] = sm.op + (BE + wq * (BQ / WQ) + mq * 32 + (lane & 31)) * ROWB;

    if (t_begin < t_end) load_stage(t_begin, 0);

    for (int64_t t = t_begin; t < t_end; ++t) {
        f32x16 acc[P::MQ][P::ME];
#pragma unroll
        for (int mq = 0; mq < P::MQ; ++mq)
#pragma unroll
            for (int me = 0; me < P::ME; ++me)
#pragma unroll
                for (int r = 0; r < 16; ++r) acc[mq][me][r] = 0.f;

        for (int ks = 0; ks < nks; ++ks) {
            __syncthreads();
#pragma unroll
            for (int j = 0; j < P::NCH; ++j) {
                const int c = tid + j * P::NT;
                *reinterpret_cast<uint4*>(sm.op + (c / (KB / 16)) * ROWB + (c % (KB / 16)) * 16) = pre[j];
            }
            __syncthreads();
            if (ks + 1 < nks) load_stage(t, ks + 1);
            else if (t + 1 < t_end) load_stage(t + 1, 0);
#pragma unroll
            for (int s = 0; s < M::NSTEP; ++s) {
                typename M::Frag fa[P::ME], fb[P::MQ];
#pragma unroll
                for (int me = 0; me < P::ME; ++me) fa[me] = M::load(a_row[me], s, h);
#pragma unroll
                for (int mq = 0; mq < P::MQ; ++mq) fb[mq] = M::load(b_row[mq], s, h);
#pragma unroll
                for (int mq = 0; mq < P::MQ; ++mq)
#pragma unroll
                    for (int me = 0; me < P::ME; ++me) M::mma(acc[mq][me], fa[me], fb[mq]);
            }
        }

        // ---- epilogue: scores, threshold test, candidate rounds ----
        // lane holds, for block (mq, me), query column wq*BQ/WQ + mq*32 + lane%32 and
        // entry rows we*BE/WE + me*32 + 8*(r/4) + 4*h + r%4, r = 0..15.
        const int64_t e_tile = t * BE + we * (BE / WE);
        float ts[P::MQ];
        int ti[P::MQ];
        float fqv[P::MQ];
        int qloc[P::MQ];
#pragma unroll
        for (int mq = 0; mq < P::MQ; ++mq) {
            qloc[mq] = wq * (BQ / WQ) + mq * 32 + (lane & 31);
            ts[mq] = sm.thr_s[qloc[mq]];
            ti[mq] = sm.thr_i[qloc[mq]];
            fqv[mq] = sm.fq[qloc[mq]];
        }
        uint64_t pend = 0;
#pragma unroll
        for (int me = 0; me < P::ME; ++me)
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                const int64_t ebase = e_tile + me * 32 + 8 * g + 4 * h;
                const float4 f4 = *reinterpret_cast<const float4*>(fe + ebase);
                const float fev[4] = {f4.x, f4.y, f4.z, f4.w};
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const int r = 4 * g + j;
                    const int64_t e = ebase + j;
#pragma unroll
                    for (int mq = 0; mq < P::MQ; ++mq) {
                        float s = acc[mq][me][r] * fev[j] * fqv[mq];
                        s = __builtin_fminf(__builtin_fmaxf(s, -1.f), 1.f);
                        acc[mq][me][r] = s;
                        const bool ok = e < n && fqv[mq] == fqv[mq] && before(s, (int)e, ts[mq], ti[mq]);
                        pend |= (uint64_t)ok << ((mq * P::ME + me) * 16 + r);
                    }
                }
            }

        int any = __syncthreads_or(pend != 0);
        while (any) {
            if (pend) {
#pragma unroll
                for (int mq = 0; mq < P::MQ; ++mq)
#pragma unroll
                    for (int me = 0; me < P::ME; ++me)
#pragma unroll
                        for (int r = 0; r < 16; ++r) {
                            const int bit = (mq * P::ME + me) * 16 + r;
                            if ((pend >> bit) & 1) {
                                const int e = (int)(e_tile + me * 32 + 8 * (r >> 2) + 4 * h + (r & 3));
                                const float s = acc[mq][me][r];
                                const int qi = qloc[mq];
                                if (!before(s, e, sm.thr_s[qi], sm.thr_i[qi])) {
                                    pend &= ~(1ull << bit);
                                } else {
                                    const int pos = atomicAdd(&sm.cnt[qi], 1);
                                    if (pos < NCAND) {
                                        sm.cand_s[qi * NCAND + pos] = s;
                                        sm.cand_i[qi * NCAND + pos] = e;
                                        pend &= ~(1ull << bit);
                                    }
                                }
                            }
                        }
            }
            __syncthreads();
            for (int qi = tid; qi < BQ; qi += P::NT) {
                int c = sm.cnt[qi];
                if (c == 0) continue;
                c = c < NCAND ? c : NCAND;
                float tsv = sm.thr_s[qi];
                int tiv = sm.thr_i[qi];
                for (int j = 0; j < c; ++j) {
                    const float s = sm.cand_s[qi * NCAND + j];
                    const int e = sm.cand_i[qi * NCAND + j];
                    if (!before(s, e, tsv, tiv)) continue;
                    int p = k - 1;
                    while (p > 0 && before(s, e, sm.list_s[(p - 1) * BQ + qi], sm.list_i[(p - 1) * BQ + qi])) {
                        sm.list_s[p * BQ + qi] = sm.list_s[(p - 1) * BQ + qi];
                        sm.list_i[p * BQ + qi] = sm.list_i[(p - 1) * BQ + qi];
                        --p;
                    }
                    sm.list_s[p * BQ + qi] = s;
                    sm.list_i[p * BQ + qi] = e;
                    tsv = sm.list_s[(k - 1) * BQ + qi];
                    tiv = sm.list_i[(k - 1) * BQ + qi];
                }
                sm.thr_s[qi] = tsv;
                sm.thr_i[qi] = tiv;
                sm.cnt[qi] = 0;
            }
            any = __syncthreads_or(pend != 0);
        }
    }

    __syncthreads();
    for (int i = tid; i < BQ * k; i += P::NT) {
        const int qi = i / k, p = i % k;
        const int64_t o = (((int64_t)q0 + qi) * splits + split) * k + p;
        part_s[o] = sm.list_s[p * BQ + qi];
        part_i[o] = sm.list_i[p * BQ + qi];
    }
}

// ---- merge of the per-split partial lists ----------------------------------
// (score, index) as one key ordered like (score desc, index asc): the score's
// bits mapped to an order-preserving unsigned integer, then the complement of
// the index.  Adding +0 turns -0 into +0, which compare equal as scores.
__device__ inline uint64_t merge_key(float s, int i)
{
    const uint32_t u = __float_as_uint(s + 0.0f);
    const uint32_t o = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
    return ((uint64_t)o << 32) | (uint32_t)~(uint32_t)i;
}
__device__ inline float merge_key_score(uint64_t key)
{
    const uint32_t o = (uint32_t)(key >> 32);
    return __uint_as_float((o & 0x80000000u) ? (o & 0x7fffffffu) : ~o);
}
// one step of a wavefront maximum: the key of the lane that the DPP control
// names (own key where it names none, or the row is masked off)
template <int CTRL, int ROWS>
__device__ inline uint64_t dpp_max_step(uint64_t v)
{
    const int lo = (int)(uint32_t)v, hi = (int)(uint32_t)(v >> 32);
    const uint32_t olo = (uint32_t)__builtin_amdgcn_update_dpp(lo, lo, CTRL, ROWS, 0xf, false);
    const uint32_t ohi = (uint32_t)__builtin_amdgcn_update_dpp(hi, hi, CTRL, ROWS, 0xf, false);
    const uint64_t o = ((uint64_t)ohi << 32) | olo;
    return o > v ? o : v;
}
// largest key of the wavefront, in every lane: quads (xor 1, xor 2), half
// rows (mirror), rows (mirror), then rows 1 and 3 take row 0's and row 2's
// maximum (broadcast of lane 15) and rows 2 and 3 row 1's (lane 31): lane 63
// ends with the maximum of all 64 lanes
__device__ inline uint64_t wave_max_key(uint64_t v)
{
    v = dpp_max_step<0xB1, 0xf>(v);      // quad_perm [1, 0, 3, 2]
    v = dpp_max_step<0x4E, 0xf>(v);      // quad_perm [2, 3, 0, 1]
    v = dpp_max_step<0x141, 0xf>(v);     // row_half_mirror
    v = dpp_max_step<0x140, 0xf>(v);     // row_mirror
    v = dpp_max_step<0x142, 0xa>(v);     // row_bcast:15
    v = dpp_max_step<0x143, 0xc>(v);     // row_bcast:31
    const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)v, 63);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(v >> 32), 63);
    return ((uint64_t)hi << 32) | lo;
}

template <int MAXOWN>
__global__ __launch_bounds__(256) void k_topk_merge(const float* __restrict__ part_s,
                                                     const int* __restrict__ part_i, int splits,
                                                     int64_t b_pad, int32_t k, int32_t b,
                                                     const float* __restrict__ fq,
                                                     float* __restrict__ top_s, int32_t* __restrict__ top_i)
{
    const int lane = threadIdx.x & 63;
    const int64_t q = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (q >= b) return;
    const float f = fq[q];
    if (!(f == f)) {                      // invalid query row
        for (int p = lane; p < k; p += 64) {
            top_s[q * k + p] = __int_as_float(0x7fc00000);
            top_i[q * k + p] = -1;
        }
        return;
    }
    const int ne = splits * k;                                     // this query's entries
    const float* gs = part_s + (int64_t)q * ne;
    const int* gi = part_i + (int64_t)q * ne;
    // a lane's list heads advance by loads from this query's block, which the
    // first loads bring into the vector cache
    auto fetch = [&](int l, int hd, float& sc, int& ix) {
        sc = gs[l * k + hd];
        ix = gi[l * k + hd];
    };
    int head[MAXOWN];
    float cs[MAXOWN];
    int ci[MAXOWN];
#pragma unroll
    for (int j = 0; j < MAXOWN; ++j) {
        const int l = lane + 64 * j;
        head[j] = 0;
        if (l < splits) {
            fetch(l, 0, cs[j], ci[j]);
        } else {
            cs[j] = neg_inf();
            ci[j] = IDX_NONE;
        }
    }
    for (int p = 0; p < k; ++p) {
        float bs = cs[0];
        int bi = ci[0], bj = 0;
#pragma unroll
        for (int j = 1; j < MAXOWN; ++j)
            if (before(cs[j], ci[j], bs, bi)) { bs = cs[j]; bi = ci[j]; bj = j; }
        const uint64_t wk = wave_max_key(merge_key(bs, bi));
        const float ws = merge_key_score(wk);
        const int wi = (int)~(uint32_t)wk;
        if (lane == 0) {
            top_s[q * k + p] = ws;
            top_i[q * k + p] = wi == IDX_NONE ? -1 : wi;
        }
        if (wi != IDX_NONE && bi == wi) {          // entry indices are unique: one owner
#pragma unroll
            for (int j = 0; j < MAXOWN; ++j)
                if (j == bj) {
                    ++head[j];
                    const int l = lane + 64 * j;
                    if (head[j] < k) {
                        fetch(l, head[j], cs[j], ci[j]);
                    } else {
                        cs[j] = neg_inf();
                        ci[j] = IDX_NONE;
                    }
                }
        }
    }
}

// variants: (BQ, BE, WQ, WE) = (128, 128, 2, 2), list capacity KMAX
template <int DT, int KMAX>
hipError_t run_simtopk(const MatchPlan& p, int64_t n, const void* emb, const float* fe,
                       const void* q, const float* fq, int32_t b, int64_t row_bytes, int32_t k,
                       float* ps, int* pi, hipStream_t s)
{
    const dim3 grid(p.splits, p.qtiles), block(256);
    k_simtopk<DT, 128, 128, 2, 2, KMAX><<<grid, block, 0, s>>>(
        static_cast<const uint8_t*>(emb), fe, n, static_cast<const uint8_t*>(q), fq, b, row_bytes,
        k, p.splits, p.b_pad, ps, pi);
    return hipGetLastError();
}

template <int DT>
hipError_t run_simtopk_k(const MatchPlan& p, int64_t n, const void* emb, const float* fe,
                         const void* q, const float* fq, int32_t b, int64_t row_bytes, int32_t k,
                         float* ps, int* pi, hipStream_t s)
{
    if (k <= 16) return run_simtopk<DT, 16>(p, n, emb, fe, q, fq, b, row_bytes, k, ps, pi, s);
    if (k <= 32) return run_simtopk<DT, 32>(p, n, emb, fe, q, fq, b, row_bytes, k, ps, pi, s);
    return run_simtopk<DT, 64>(p, n, emb, fe, q, fq, b, row_bytes, k, ps, pi, s);
}

inline size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

}  // namespace

MatchPlan plan_match(int dt, int64_t n, int32_t d, int32_t b, int32_t k)
{
    MatchPlan p{};
    const int64_t rb = (int64_t)d * elem_bytes(dt);
    const int64_t group = dt == APC_E4M3 ? 6 * 128 : 4 * 128;   // chunks in flight x 128 bytes
    const int q2b = qs_queries(dt, rb, k);
    const int q8b = qs8_queries(dt, rb, k);
    if (q8b > 0 && b > 256) {
        // large batches of 512- or 768-byte rows: two wavefronts per SIMD,
        // 256 queries per workgroup, one workgroup per CU
        p.kernel = KERNEL_QS8;
        p.bq = q8b;
        p.qtiles = (b + p.bq - 1) / p.bq;
        const int64_t ngr = (n + qs8_group_rows() - 1) / qs8_group_rows();
        int64_t splits = p.qtiles >= 256 ? 1 : 256 / p.qtiles;
        if (splits > ngr) splits = ngr;
        if (splits < 1) splits = 1;
        p.splits = (int)splits;
    } else if (q2b > 0 && k <= qs_max_k()) {
        // 16-bit or e4m3 rows: queries in VGPRs, cache rows through LDS, one
        // workgroup per CU; the query tiles of a split share an XCD
        p.kernel = KERNEL_QS;
        p.bq = q2b;
        p.qtiles = (b + p.bq - 1) / p.bq;
        if (p.qtiles < 1) p.qtiles = 1;
        const int64_t gr = qs_group_rows(rb, k);
        const int64_t ngr = (n + gr - 1) / gr;
        int64_t splits = p.qtiles >= 256 ? 1 : 256 / p.qtiles;
        if (splits > ngr) splits = ngr;
        if (splits < 1) splits = 1;
        p.splits = (int)splits;
    } else if (f32s_fits(dt, n, d, b, k)) {
        // small float32 caches: a workgroup per 32-row block, d over its wavefronts
        p.kernel = KERNEL_F32S;
        p.bq = f32s_queries();
        p.qtiles = (b + p.bq - 1) / p.bq;
        p.splits = (int)((n + f32s_rows() - 1) / f32s_rows());
    } else if (b <= 256 && rb <= 3072 && rb % group == 0) {
        // small batch: query tile resident in LDS, entries streamed from HBM
        const bool wide = k <= 16 && rb <= 1536 && dt != APC_E4M3;
        p.kernel = wide ? KERNEL_STREAM_64 : KERNEL_STREAM_32;
        p.bq = wide ? 64 : 32;
        p.qtiles = (b + p.bq - 1) / p.bq;
        if (p.qtiles < 1) p.qtiles = 1;
        const int64_t nblk = (n + 31) / 32;
        int64_t splits = (256 + p.qtiles - 1) / p.qtiles;   // one workgroup per CU
        if (splits > nblk) splits = nblk;
        if (splits > 512) splits = 512;
        if (splits < 1) splits = 1;
        p.splits = (int)splits;
    } else {
        p.kernel = KERNEL_TILED;
        p.bq = 128;
        p.qtiles = (b + p.bq - 1) / p.bq;
        if (p.qtiles < 1) p.qtiles = 1;
        const int64_t ntiles = (n + 127) / 128;
        const int target = k <= 16 ? 512 : 256;      // resident workgroups across 256 CUs
        int64_t splits = (target + p.qtiles - 1) / p.qtiles;
        if (splits > ntiles) splits = ntiles;
        if (splits > 512) splits = 512;
        if (splits < 1) splits = 1;
        p.splits = (int)splits;
    }
    p.b_pad = (int64_t)p.qtiles * p.bq;
    p.off_fq = 0;
    p.off_gt = align256(p.off_fq + sizeof(float) * (size_t)p.b_pad);
    // the two-wavefront kernel's per-split quantile scores (splits x b_pad)
    p.off_g2 = align256(p.off_gt + sizeof(int) * (size_t)p.b_pad);
    const size_t g2_bytes = p.kernel == KERNEL_QS8 ? sizeof(int) * (size_t)p.splits * p.b_pad : 0;
    p.off_ps = align256(p.off_g2 + g2_bytes);
    p.off_pi = align256(p.off_ps + sizeof(float) * (size_t)p.splits * p.b_pad * k);
    p.off_qp = align256(p.off_pi + sizeof(int) * (size_t)p.splits * p.b_pad * k);
    const size_t qp_bytes =
        p.kernel == KERNEL_QS || p.kernel == KERNEL_QS8 ? (size_t)p.b_pad * (size_t)d * elem_bytes(dt) : 0;
    p.bytes = align256(p.off_qp + qp_bytes);
    return p;
}

hipError_t launch_match(const MatchPlan& p, int dt, int64_t n, int32_t d, const void* emb,
                        const float* fe, const void* q, const float* q_scale, int32_t b, int32_t k,
                        float* top_score, int32_t* top_idx, void* ws, hipStream_t s,
                        hipEvent_t ev_start, hipEvent_t ev_stop)
{
    uint8_t* w = static_cast<uint8_t*>(ws);
    float* fq = reinterpret_cast<float*>(w + p.off_fq);
    float* ps = reinterpret_cast<float*>(w + p.off_ps);
    int* pi = reinterpret_cast<int*>(w + p.off_pi);
    const int64_t row_bytes = (int64_t)d * elem_bytes(dt);

    hipError_t e;
    if (p.kernel == KERNEL_TILED) {
        if ((e = launch_row_factors(dt, b, d, q, q_scale, nullptr, 0, fq, nullptr, s)) != hipSuccess) return e;
        if (ev_start && (e = hipEventRecord(ev_start, s)) != hipSuccess) return e;
        switch (dt) {
        case APC_F32: e = run_simtopk_k<APC_F32>(p, n, emb, fe, q, fq, b, row_bytes, k, ps, pi, s); break;
        case APC_F16: e = run_simtopk_k<APC_F16>(p, n, emb, fe, q, fq, b, row_bytes, k, ps, pi, s); break;
        case APC_BF16: e = run_simtopk_k<APC_BF16>(p, n, emb, fe, q, fq, b, row_bytes, k, ps, pi, s); break;
        default: e = run_simtopk_k<APC_E4M3>(p, n, emb, fe, q, fq, b, row_bytes, k, ps, pi, s); break;
        }
    } else if (p.kernel == KERNEL_F32S) {
        if ((e = launch_row_factors(dt, b, d, q, q_scale, nullptr, 0, fq, nullptr, s)) != hipSuccess) return e;
        if (ev_start && (e = hipEventRecord(ev_start, s)) != hipSuccess) return e;
        e = launch_f32s(p, n, d, emb, fe, q, fq, b, k, ps, pi, s);
    } else if (p.kernel == KERNEL_QS) {
        int* gt = reinterpret_cast<int*>(w + p.off_gt);
        uint8_t* qp = w + p.off_qp;
        if ((e = launch_qprep(dt, q, q_scale, b, p.b_pad, row_bytes, fq, gt, qp, p.bq, 4, nullptr, 0, s)) != hipSuccess)
            return e;
        if (ev_start && (e = hipEventRecord(ev_start, s)) != hipSuccess) return e;
        e = launch_qs(p, dt, n, d, emb, fe, qp, fq, gt, b, k, ps, pi, s);
    } else if (p.kernel == KERNEL_QS8) {
        int* gt = reinterpret_cast<int*>(w + p.off_gt);
        uint8_t* qp = w + p.off_qp;
        int* g2 = reinterpret_cast<int*>(w + p.off_g2);
        if ((e = launch_qprep(dt, q, q_scale, b, p.b_pad, row_bytes, fq, gt, qp, p.bq, 8, g2, p.splits, s)) != hipSuccess)
            return e;
        if (ev_start && (e = hipEventRecord(ev_start, s)) != hipSuccess) return e;
        e = launch_qs8(p, dt, n, d, emb, fe, qp, fq, gt, g2, b, k, ps, pi, s);
    } else {
        if (ev_start && (e = hipEventRecord(ev_start, s)) != hipSuccess) return e;
        e = launch_stream(p, dt, n, d, emb, fe, q, q_scale, b, k, fq, ps, pi, s);
    }
    if (e != hipSuccess) return e;
    if (ev_stop && (e = hipEventRecord(ev_stop, s)) != hipSuccess) return e;
    const dim3 grid((unsigned)((b + 3) / 4)), block(256);
    if (p.splits <= 64)
        k_topk_merge<1><<<grid, block, 0, s>>>(ps, pi, p.splits, p.b_pad, k, b, fq, top_score, top_idx);
    else if (p.splits <= 128)
        k_topk_merge<2><<<grid, block, 0, s>>>(ps, pi, p.splits, p.b_pad, k, b, fq, top_score, top_idx);
    else if (p.splits <= 256)
        k_topk_merge<4><<<grid, block, 0, s>>>(ps, pi, p.splits, p.b_pad, k, b, fq, top_score, top_idx);
    else
        k_topk_merge<8><<<grid, block, 0, s>>>(ps, pi, p.splits, p.b_pad, k, b, fq, top_score, top_idx);
    return hipGetLastError();
}

}  // namespace apc
