// Latent gather: copy the cached latent of each placed query's nearest entry
// into its (instance, slot) of the batch buffer.  A slot holds lps latents:
// one for every level (lps = 1), or one per level 1..lps, level-major inside
// the slot (pool row slot * lps + level - 1).  One workgroup per query,
// 16-byte loads and stores spread over the workgroup so every wavefront
// moves 1 KiB contiguous per instruction.
#include "apc_internal.h"

namespace apc {
namespace {

__global__ __launch_bounds__(256) void k_gather(const uint8_t* __restrict__ pool, int64_t n_entries,
                                                int64_t n_slots, int64_t latent_bytes,
                                                const int32_t* __restrict__ slot_of_entry,
                                                const int32_t* __restrict__ top_idx, int32_t ld,
                                                const int32_t* __restrict__ out_level,
                                                const int32_t* __restrict__ out_inst,
                                                const int32_t* __restrict__ out_slot, int32_t n_inst,
                                                int32_t slots_per_inst, int32_t lps,
                                                uint8_t* __restrict__ batch, int32_t* __restrict__ hit)
{
    const int64_t q = blockIdx.x;
    const int32_t e = top_idx[q * ld];
    const int32_t lvl = out_level[q], inst = out_inst[q], slot = out_slot[q];
    int64_t src = -1;
    if (lvl > 0 && (lps == 1 || lvl <= lps) && e >= 0 && e < n_entries && inst >= 0 && inst < n_inst &&
        slot >= 0 && slot < slots_per_inst) {
        src = slot_of_entry ? (int64_t)slot_of_entry[e] : (int64_t)e;
        if (src >= n_slots / lps) src = -1;
        else if (src >= 0 && lps > 1) src = src * lps + (lvl - 1);
    }
    if (threadIdx.x == 0) hit[q] = src >= 0 ? 1 : 0;
    if (src < 0) return;
    const uint4* s = reinterpret_cast<const uint4*>(pool + src * latent_bytes);
    uint4* d = reinterpret_cast<uint4*>(batch + ((int64_t)inst * slots_per_inst + slot) * latent_bytes);
    const int64_t nv = latent_bytes / 16;
    for (int64_t c = threadIdx.x; c < nv; c += 256) d[c] = s[c];
}

}  // namespace

hipError_t launch_gather(const void* pool, int64_t n_entries, int64_t n_slots, int64_t latent_bytes,
                         const int32_t* slot_of_entry, const int32_t* top_idx, int32_t ld, int32_t b,
                         const int32_t* out_level, const int32_t* out_inst, const int32_t* out_slot,
                         int32_t n_inst, int32_t slots_per_inst, int32_t lps, void* batch, int32_t* hit,
                         hipStream_t s)
{
    if (b <= 0) return hipSuccess;
    k_gather<<<(unsigned)b, 256, 0, s>>>(static_cast<const uint8_t*>(pool), n_entries, n_slots,
                                         latent_bytes, slot_of_entry, top_idx, ld, out_level, out_inst,
                                         out_slot, n_inst, slots_per_inst, lps, static_cast<uint8_t*>(batch), hit);
    return hipGetLastError();
}

}  // namespace apc
