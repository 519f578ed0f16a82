// Query preparation for the query-stationary kernels and their dispatch by
// storage type (the kernels are in qs_kernel.h and qs8_kernel.h, instantiated
// per type).
#include "qs8_kernel.h"

namespace apc {
namespace {

// query factors f = 1/|q| (NaN for rows that cannot be matched: non-finite,
// zero norm, bad e4m3 scale, or padding) and reset global bounds, one
// wavefront per padded query row.  The row's 16-byte units also go to qperm
// in the order the kernel loads them (zeros for padding rows): with nw
// wavefronts per query tile of bq rows, row r of tile r / bq is query block
// mq of wavefront w in that tile, lane h 32 + r % 32 loads at its step s the
// units of byte offsets 128 (s UPS / 4) + 64 h + 16 ((s UPS + i) % 4),
// i < UPS, and those sit at unit ((((tile nw + w) MQ + mq) QST + s) 64 +
// lane) UPS + i of qperm, so that a wavefront's load of one step reads 64 UPS
// consecutive units.
template <int DT>
__global__ __launch_bounds__(256) void k_qprep(const uint8_t* __restrict__ qry, const float* __restrict__ q_scale,
                                                int32_t b, int64_t b_pad, int64_t row_bytes,
                                                float* __restrict__ fq, int* __restrict__ gthr,
                                                uint8_t* __restrict__ qperm, int bq, int nw, int* __restrict__ g2, int nsplit)
{
    constexpr int UPS = Q2Op<DT>::UPS;
    const int lane = threadIdx.x & 63;
    const int64_t r = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (r >= b_pad) return;
    const int bqw = bq / nw, mqn = bqw / 32;                   // queries per wavefront, blocks
    const int64_t tile = r / bq;
    const int local = (int)(r - tile * bq);
    const int w = local / bqw, mq = (local % bqw) / 32, r32 = local & 31;
    const int64_t qst = row_bytes / (32 * UPS);
    uint8_t* tp = qperm + ((((tile * nw + w) * mqn + mq) * qst) * 64 + r32) * (UPS * 16);
    float ss = 0.f;
    bool bad = false;
    const uint8_t* row = qry + r * row_bytes;
    constexpr int U = 2;                                           // units per lane in flight
    for (int64_t off0 = (int64_t)lane * 16; off0 < row_bytes; off0 += U * 64 * 16) {
        uint4 v[U];
#pragma unroll
        for (int i = 0; i < U; ++i) {
            const int64_t off = off0 + i * 64 * 16;
            v[i] = make_uint4(0u, 0u, 0u, 0u);
            if (r < b && off < row_bytes) v[i] = *reinterpret_cast<const uint4*>(row + off);
        }
#pragma unroll
        for (int i = 0; i < U; ++i) {
            const int64_t off = off0 + i * 64 * 16;
            if (off >= row_bytes) continue;
            if (r < b) sumsq16<DT>(v[i], ss, bad);
            const int64_t u = (off >> 7) * 4 + ((off >> 4) & 3);  // unit within its half-row order
            const int h = (int)((off >> 6) & 1);
            const int64_t st = u / UPS, piece = u % UPS;
            *reinterpret_cast<uint4*>(tp + (st * 64 + h * 32) * (UPS * 16) + piece * 16) = v[i];
        }
    }
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) ss += __shfl_xor(ss, m, 64);
    bad = __any(bad);
    if (g2)
        for (int sp = lane; sp < nsplit; sp += 64) g2[(int64_t)sp * b_pad + r] = q2_key(neg_inf());
    if (lane != 0) return;
    bool ok = r < b && !bad && __builtin_isfinite(ss) && ss > 0.f;
    if (ok && q_scale) {
        const float sc = q_scale[r];
        ok = __builtin_isfinite(sc) && sc > 0.f;
    }
    fq[r] = ok ? 1.0f / __builtin_sqrtf(ss) : qnan();
    gthr[r] = q2_key(neg_inf());
}

}  // namespace

int qs_queries(int dt, int64_t row_bytes, int k)
{
    return dt == APC_F16 || dt == APC_BF16 || dt == APC_E4M3 ? q2_queries(row_bytes, k) : 0;
}

int qs_max_k() { return Q2_KMAX; }

int qs_group_rows(int64_t row_bytes, int k) { return q2_rows(row_bytes, k); }

int qs8_queries(int dt, int64_t row_bytes, int k)
{
    return (dt == APC_F16 || dt == APC_BF16 || dt == APC_E4M3) && q8_built(row_bytes, k) ? Q8_NW * 32 : 0;
}

int qs8_group_rows() { return Q8_GR; }

hipError_t launch_qprep(int dt, const void* q, const float* q_scale, int32_t b, int64_t b_pad, int64_t row_bytes,
                        float* fq, int* gthr, uint8_t* qperm, int bq, int nw, int* g2, int nsplit, hipStream_t s)
{
    const dim3 grid((unsigned)((b_pad + 3) / 4)), block(256);
    const uint8_t* qp = static_cast<const uint8_t*>(q);
    switch (dt) {
    case APC_F16: k_qprep<APC_F16><<<grid, block, 0, s>>>(qp, q_scale, b, b_pad, row_bytes, fq, gthr, qperm, bq, nw, g2, nsplit); break;
    case APC_BF16: k_qprep<APC_BF16><<<grid, block, 0, s>>>(qp, q_scale, b, b_pad, row_bytes, fq, gthr, qperm, bq, nw, g2, nsplit); break;
    case APC_E4M3: k_qprep<APC_E4M3><<<grid, block, 0, s>>>(qp, q_scale, b, b_pad, row_bytes, fq, gthr, qperm, bq, nw, g2, nsplit); break;
    default: return hipErrorInvalidValue;                          // the query-stationary kernels take 16-bit or e4m3 rows
    }
    return hipGetLastError();
}

hipError_t launch_qs(const MatchPlan& p, int dt, int64_t n, int32_t d, const void* emb, const float* fe,
                     const void* q, const float* fq, int* gthr, int32_t b, int32_t k, float* ps, int* pi,
                     hipStream_t s)
{
    const int64_t rb = (int64_t)d * elem_bytes(dt);
    switch (dt) {
    case APC_F16: return launch_qs_f16(p, n, rb, emb, fe, q, fq, gthr, b, k, ps, pi, s);
    case APC_BF16: return launch_qs_bf16(p, n, rb, emb, fe, q, fq, gthr, b, k, ps, pi, s);
    case APC_E4M3: return launch_qs_e4m3(p, n, rb, emb, fe, q, fq, gthr, b, k, ps, pi, s);
    default: return hipErrorInvalidValue;
    }
}

hipError_t launch_qs8(const MatchPlan& p, int dt, int64_t n, int32_t d, const void* emb, const float* fe,
                      const void* q, const float* fq, int* gthr, int* g2, int32_t b, int32_t k, float* ps, int* pi,
                      hipStream_t s)
{
    const int64_t rb = (int64_t)d * elem_bytes(dt);
    switch (dt) {
    case APC_F16: return launch_qs8_f16(p, n, rb, emb, fe, q, fq, gthr, g2, b, k, ps, pi, s);
    case APC_BF16: return launch_qs8_bf16(p, n, rb, emb, fe, q, fq, gthr, g2, b, k, ps, pi, s);
    case APC_E4M3: return launch_qs8_e4m3(p, n, rb, emb, fe, q, fq, gthr, g2, b, k, ps, pi, s);
    default: return hipErrorInvalidValue;
    }
}

}  // namespace apc
