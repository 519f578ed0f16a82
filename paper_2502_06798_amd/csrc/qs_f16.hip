// Instantiations of the query-stationary similarity + top-k kernel for f16 rows.
#include "qs_kernel.h"

namespace apc {

hipError_t launch_qs_f16(const MatchPlan& p, int64_t n, int64_t rb, const void* emb, const float* fe, const void* q,
                         const float* fq, int* gthr, int32_t b, int32_t k, float* ps, int* pi, hipStream_t s)
{
    if (rb == 1536) return run_qs<APC_F16, 1536, 1>(p, n, emb, fe, q, fq, gthr, b, k, ps, pi, s);
    if (rb == 1024) return run_qs<APC_F16, 1024, 2>(p, n, emb, fe, q, fq, gthr, b, k, ps, pi, s);
    if (rb == 768) return run_qs<APC_F16, 768, 2>(p, n, emb, fe, q, fq, gthr, b, k, ps, pi, s);
    if (rb == 512) return run_qs<APC_F16, 512, 2>(p, n, emb, fe, q, fq, gthr, b, k, ps, pi, s);
    return hipErrorInvalidValue;
}

}  // namespace apc
