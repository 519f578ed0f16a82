// Instantiations of the two-wavefronts-per-SIMD similarity + top-k kernel for f16 rows.
#include "qs8_kernel.h"

namespace apc {

hipError_t launch_qs8_f16(const MatchPlan& p, int64_t n, int64_t rb, const void* emb, const float* fe, const void* q,
                         const float* fq, int* gthr, int* g2, int32_t b, int32_t k, float* ps, int* pi, hipStream_t s)
{
    return q8_dispatch<APC_F16>(p, n, rb, emb, fe, q, fq, gthr, g2, b, k, ps, pi, s);
}

}  // namespace apc
