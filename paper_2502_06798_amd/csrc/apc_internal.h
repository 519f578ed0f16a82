// Internal declarations shared by the host library and the kernel files.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "../../include/apc.h"

namespace apc {

inline int elem_bytes(int dt)
{
    switch (dt) {
    case APC_F32: return 4;
    case APC_F16: case APC_BF16: return 2;
    case APC_E4M3: return 1;
    default: return 0;
    }
}

// ---- row factors (cache build and query preparation) ----------------------
// bits of the build status word
enum : uint32_t { ST_NONFINITE = 1u, ST_ZERO = 2u, ST_SCALE = 4u, ST_SLOT = 8u };
struct BuildStatus {
    uint32_t flags;
    uint32_t pad;
    unsigned long long first_bad;   // lowest bad row (or entry) index
    unsigned long long n_bad;       // bad rows (or entries)
};

// f[r] = 1/|row r| (NaN for bad rows; f may be null); when st != nullptr
// also records bad rows, non-positive or non-finite scales and out-of-range
// slots; when rowflags != nullptr writes each row's ST_ bits there.
hipError_t launch_row_factors(int dt, int64_t n, int32_t d, const void* rows, const float* scale,
                              const int32_t* slot_of_entry, int64_t n_slots, float* f,
                              BuildStatus* st, hipStream_t s, uint8_t* rowflags = nullptr);

// float32 rows to a storage type (f16/bf16 rounded to nearest-even; e4m3fn
// codes with a per-row scale amax / 448 and a clamp to +-448)
hipError_t launch_quantize_rows(int dt, int64_t n, int32_t d, const float* x, void* out, float* scale,
                                hipStream_t s);

// factor layout of a cache: n rounded up to a multiple of 256 factors, zeros past n
__host__ __device__ inline int64_t factor_pad(int64_t n) { return (n + 255) / 256 * 256; }

// ---- similarity + top-k ----------------------------------------------------
enum { KERNEL_TILED = 0, KERNEL_STREAM_64 = 1, KERNEL_STREAM_32 = 2, KERNEL_QS = 4, KERNEL_QS8 = 5, KERNEL_F32S = 6 };
struct MatchPlan {
    int kernel;        // kernel variant id
    int bq;            // queries per workgroup tile
    int qtiles;        // ceil(b / bq)
    int splits;        // workgroups along the entries per query tile
    int64_t b_pad;     // qtiles * bq
    size_t off_fq, off_gt, off_g2, off_ps, off_pi, off_qp, bytes;   // workspace layout
};
MatchPlan plan_match(int dt, int64_t n, int32_t d, int32_t b, int32_t k);

// ev_start/ev_stop (may be null) are recorded around the similarity kernel.
hipError_t launch_match(const MatchPlan& p, int dt, int64_t n, int32_t d, const void* emb,
                        const float* fe, const void* q, const float* q_scale, int32_t b, int32_t k,
                        float* top_score, int32_t* top_idx, void* ws, hipStream_t s,
                        hipEvent_t ev_start, hipEvent_t ev_stop);

// streaming kernel for small batches (query factors are computed inside and
// written to fq by the first split)
hipError_t launch_stream(const MatchPlan& p, int dt, int64_t n, int32_t d, const void* emb,
                         const float* fe, const void* q, const float* q_scale, int32_t b, int32_t k,
                         float* fq, float* ps, int* pi, hipStream_t s);

// query-stationary kernel for 16-bit and e4m3 rows of 512, 768, 1024 or 1536 bytes (k <= qs_max_k()):
// queries in VGPRs, cache rows through an LDS ring, per-query bounds shared
// between workgroups.  qs_queries gives the queries per workgroup (0: not built).
int qs_queries(int dt, int64_t row_bytes, int k);
int qs_max_k();
// entries per group (the unit a split is made of) of the shape qs_queries describes
int qs_group_rows(int64_t row_bytes, int k);
// query factors into fq and reset bounds gthr, for b_pad rows (rows >= b get NaN)
// query factors and bound reset for the query-stationary kernels; qperm
// (b_pad x row_bytes bytes) receives the queries in the order that kernel's
// lanes load them, for query tiles of bq rows over nw wavefronts
hipError_t launch_qprep(int dt, const void* q, const float* q_scale, int32_t b, int64_t b_pad, int64_t row_bytes,
                        float* fq, int* gthr, uint8_t* qperm, int bq, int nw, int* g2, int nsplit, hipStream_t s);
hipError_t launch_qs(const MatchPlan& p, int dt, int64_t n, int32_t d, const void* emb, const float* fe,
                     const void* q, const float* fq, int* gthr, int32_t b, int32_t k, float* ps, int* pi,
                     hipStream_t s);
// the same with two wavefronts per SIMD and the top-k lists in LDS, for
// 16-bit and e4m3 rows of 512, 768 or 1024 bytes (k <= 32): qs8_queries gives the
// queries per workgroup (0: not built), qs8_group_rows the rows per group
int qs8_queries(int dt, int64_t row_bytes, int k);
int qs8_group_rows();
hipError_t launch_qs8(const MatchPlan& p, int dt, int64_t n, int32_t d, const void* emb, const float* fe,
                      const void* q, const float* fq, int* gthr, int* g2, int32_t b, int32_t k, float* ps, int* pi,
                      hipStream_t s);

// float32 caches of at most 512 blocks of 32 rows, d a multiple of 64, k <= 32,
// b <= 256: one workgroup per 32-row block and 16-query tile, four wavefronts
// over d (f32small.hip); the query factors come first from launch_row_factors
bool f32s_fits(int dt, int64_t n, int32_t d, int32_t b, int32_t k);
int f32s_queries();
int f32s_rows();
hipError_t launch_f32s(const MatchPlan& p, int64_t n, int32_t d, const void* emb, const float* fe, const void* q,
                       const float* fq, int32_t b, int32_t k, float* ps, int* pi, hipStream_t s);

// ---- assignment ------------------------------------------------------------
struct AssignTable {
    int32_t L;
    int32_t n_inst;
    float theta[APC_MAX_LEVELS];
    int32_t K[APC_MAX_LEVELS + 1];               // skipped steps per level, K[0] = 0
    int32_t level_cap[APC_MAX_LEVELS + 1];       // places per level
    int32_t level_first[APC_MAX_LEVELS + 2];     // first ordered instance of each level
    int16_t ord_inst[APC_MAX_INST];              // instances by (level, queue desc, index asc)
    int32_t ord_cum[APC_MAX_INST];               // places of earlier instances of the same level
    int32_t ord_cap[APC_MAX_INST];
};

hipError_t launch_assign(const AssignTable& t, const float* top_score, int32_t ld, int32_t b,
                         int32_t* opt_level, int32_t* out_level, int32_t* out_inst,
                         int32_t* out_slot, int32_t* inst_fill, hipStream_t s);

// Placement that follows a route plan (planned: computed in the kernel from
// the batch's level histogram and written to plan; else read from plan).
hipError_t launch_assign_plan(const AssignTable& t, bool planned, const float* top_score, int32_t ld, int32_t b,
                              int32_t* plan, int32_t* opt_level, int32_t* out_level, int32_t* out_inst,
                              int32_t* out_slot, int32_t* inst_fill, hipStream_t s);

// ---- resident-aware fallback, level histogram ----
hipError_t launch_resident_best(const int32_t* slot_of_entry, int64_t n_entries, int64_t n_slots,
                                const float* top_score, const int32_t* top_idx, int32_t ld, int32_t k, int32_t b,
                                float* out_score, int32_t* out_idx, hipStream_t s);
hipError_t launch_level_histogram(const int32_t* level, int32_t b, int32_t L, int32_t* hist, hipStream_t s);

// ---- merge of shard lists ----
struct ShardOffsets {
    int32_t v[APC_MAX_SHARDS];
};
hipError_t launch_merge_shards(const float* scores, const int32_t* idx, int32_t g, int32_t b, int32_t kin,
                               const ShardOffsets& off, int32_t k, float* out_s, int32_t* out_i, hipStream_t s);

// ---- gather ----------------------------------------------------------------
hipError_t launch_gather(const void* pool, int64_t n_entries, int64_t n_slots, int64_t latent_bytes,
                         const int32_t* slot_of_entry, const int32_t* top_idx, int32_t ld, int32_t b,
                         const int32_t* out_level, const int32_t* out_inst, const int32_t* out_slot,
                         int32_t n_inst, int32_t slots_per_inst, int32_t lps, void* batch, int32_t* hit,
                         hipStream_t s);

}  // namespace apc
