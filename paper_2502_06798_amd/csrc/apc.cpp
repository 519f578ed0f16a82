// C ABI of the matching library: argument checks, handle lifetime,
// workspace sizing and kernel launches on the caller's stream.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <cstdarg>
#include <climits>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <new>
#include <string>

#include "apc_internal.h"
#include "route_plan.h"

struct apc_cache {
    apc_dtype dt;
    int64_t n;
    int32_t d;
    const void* emb;
    const float* row_scale;
    const void* latents;
    int64_t n_slots;
    int64_t latent_bytes;
    const int32_t* slot_of_entry;
    float* fe;          // owned: row factors and group bounds (layout in apc_internal.h)
    int device;
};

// Workspace of apc_match_batch_static: one copy per device, held until the
// process ends.  In host code `scratch` only names the symbol; its device
// address (per device) comes from hipGetSymbolAddress.
static __device__ __align__(256) uint8_t scratch[APC_STATIC_WS_BYTES];

namespace {

constexpr int MAX_DEVICES = 64;
std::atomic<void*> g_scratch_ptr[MAX_DEVICES];   // device address of `scratch` per device (null: not looked up yet)

thread_local std::string g_err;
thread_local hipEvent_t g_ev_start = nullptr, g_ev_stop = nullptr;

apc_status fail(apc_status s, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
apc_status fail(apc_status s, const char* fmt, ...)
{
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_err = buf;
    return s;
}

apc_status ok()
{
    g_err.clear();
    return APC_OK;
}

apc_status hip_fail(hipError_t e, const char* what)
{
    return fail(APC_E_HIP, "%s: %s", what, hipGetErrorString(e));
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

bool valid_dtype(int dt) { return dt >= APC_F32 && dt <= APC_E4M3; }

apc_status check_rows(apc_dtype dt, int64_t n, int32_t d, const void* rows, const char* what)
{
    if (!valid_dtype(dt)) return fail(APC_E_DTYPE, "unknown dtype %d", (int)dt);
    if (n < 0 || d < 1) return fail(APC_E_ARG, "%s: need n >= 0 and d >= 1 (n=%lld d=%d)", what, (long long)n, d);
    if (((int64_t)d * apc::elem_bytes(dt)) % 16 != 0)
        return fail(APC_E_ARG, "%s: row of %d elements is not a multiple of 16 bytes", what, d);
    if (n > 0 && (!rows || !aligned16(rows)))
        return fail(APC_E_ARG, "%s: rows must be a non-NULL 16-byte aligned device pointer", what);
    return APC_OK;
}

// Calls that take a handle run on the handle's device: its row factors and
// the caller's borrowed buffers live there.
apc_status check_device(const char* who, const apc_cache* c)
{
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return fail(APC_E_HIP, "%s: hipGetDevice: %s", who, hipGetErrorString(e));
    if (dev != c->device)
        return fail(APC_E_ARG, "%s: the cache was built on device %d but device %d is current", who, c->device, dev);
    return APC_OK;
}

}  // namespace

extern "C" {

const char* apc_status_str(apc_status s)
{
    switch (s) {
    case APC_OK: return "ok";
    case APC_E_ARG: return "invalid argument";
    case APC_E_DTYPE: return "unknown dtype";
    case APC_E_TABLE: return "invalid threshold or instance table";
    case APC_E_NONFINITE: return "non-finite value";
    case APC_E_ZERO_NORM: return "zero-norm row";
    case APC_E_WORKSPACE: return "workspace too small";
    case APC_E_NOMEM: return "out of memory";
    case APC_E_HIP: return "HIP error";
    default: break;
    }
    return "unknown status";
}

const char* apc_last_error(void) { return g_err.c_str(); }

apc_status apc_set_kernel_events(void* start, void* stop)
{
    if ((start == nullptr) != (stop == nullptr))
        return fail(APC_E_ARG, "apc_set_kernel_events: give both events or neither");
    g_ev_start = static_cast<hipEvent_t>(start);
    g_ev_stop = static_cast<hipEvent_t>(stop);
    return ok();
}

apc_status apc_row_factors(apc_dtype dt, int64_t n, int32_t d, const void* rows, float* out, void* stream)
{
    apc_status st = check_rows(dt, n, d, rows, "apc_row_factors");
    if (st != APC_OK) return st;
    if (n > 0 && !out) return fail(APC_E_ARG, "apc_row_factors: out is NULL");
    if (n == 0) return ok();
    hipError_t e = apc::launch_row_factors(dt, n, d, rows, nullptr, nullptr, 0, out, nullptr,
                                           static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "row factor launch");
    return ok();
}

apc_status apc_quantize_rows(apc_dtype dt, int64_t n, int32_t d, const float* x, void* out, float* row_scale,
                             void* stream)
{
    if (valid_dtype(dt) && dt == APC_F32)
        return fail(APC_E_DTYPE, "apc_quantize_rows: the target must be f16, bf16 or e4m3");
    apc_status st = check_rows(dt, n, d, out, "apc_quantize_rows");
    if (st != APC_OK) return st;
    if (n > 0 && (!x || !aligned16(x)))
        return fail(APC_E_ARG, "apc_quantize_rows: x must be a non-NULL 16-byte aligned device pointer");
    if (n > 0 && (dt == APC_E4M3) != (row_scale != nullptr))
        return fail(APC_E_ARG, "apc_quantize_rows: row_scale is required for e4m3 and only for e4m3");
    if (n == 0) return ok();
    hipError_t e = apc::launch_quantize_rows(dt, n, d, x, out, row_scale, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "quantize launch");
    return ok();
}

apc_status apc_validate_rows(apc_dtype dt, int64_t n, int32_t d, const void* rows, const float* row_scale,
                             uint8_t* bad, int64_t* n_bad, int64_t* first_bad, void* stream)
{
    if (!n_bad) return fail(APC_E_ARG, "apc_validate_rows: n_bad is NULL");
    *n_bad = 0;
    if (first_bad) *first_bad = -1;
    apc_status st = check_rows(dt, n, d, rows, "apc_validate_rows");
    if (st != APC_OK) return st;
    if (n > 0 && (dt == APC_E4M3) != (row_scale != nullptr))
        return fail(APC_E_ARG, "apc_validate_rows: row_scale is required for e4m3 and only for e4m3");
    if (n == 0) return ok();
    hipStream_t s = static_cast<hipStream_t>(stream);
    apc::BuildStatus* dst = nullptr;
    apc::BuildStatus hst{};
    hst.first_bad = ~0ull;
    hipError_t e = hipMalloc(&dst, sizeof(apc::BuildStatus));
    if (e != hipSuccess) return fail(APC_E_NOMEM, "apc_validate_rows: hipMalloc: %s", hipGetErrorString(e));
    if ((e = hipMemcpyAsync(dst, &hst, sizeof hst, hipMemcpyHostToDevice, s)) != hipSuccess ||
        (e = apc::launch_row_factors(dt, n, d, rows, row_scale, nullptr, 0, nullptr, dst, s, bad)) != hipSuccess ||
        (e = hipMemcpyAsync(&hst, dst, sizeof hst, hipMemcpyDeviceToHost, s)) != hipSuccess ||
        (e = hipStreamSynchronize(s)) != hipSuccess) {
        (void)hipFree(dst);
        return hip_fail(e, "apc_validate_rows");
    }
    (void)hipFree(dst);
    *n_bad = (int64_t)hst.n_bad;
    if (first_bad) *first_bad = hst.n_bad ? (int64_t)hst.first_bad : -1;
    return ok();
}

apc_status apc_build_cache(apc_dtype dt, int64_t n, int32_t d, const void* emb, const float* row_scale,
                           const void* latents, int64_t n_slots, int64_t latent_bytes,
                           const int32_t* slot_of_entry, void* stream, apc_cache** out)
{
    if (!out) return fail(APC_E_ARG, "apc_build_cache: out is NULL");
    *out = nullptr;
    apc_status st = check_rows(dt, n, d, emb, "apc_build_cache");
    if (st != APC_OK) return st;
    if (n < 1 || n >= INT32_MAX)
        return fail(APC_E_ARG, "apc_build_cache: need 1 <= n < 2^31 - 1 entries (n=%lld)", (long long)n);
    if ((dt == APC_E4M3) != (row_scale != nullptr))
        return fail(APC_E_ARG, "apc_build_cache: row_scale is required for e4m3 and only for e4m3");
    if (n_slots < 0 || latent_bytes < 0)
        return fail(APC_E_ARG, "apc_build_cache: negative n_slots or latent_bytes");
    if (n_slots > 0) {
        if (!latents || !aligned16(latents))
            return fail(APC_E_ARG, "apc_build_cache: latents must be a 16-byte aligned device pointer");
        if (latent_bytes <= 0 || latent_bytes % 16 != 0)
            return fail(APC_E_ARG, "apc_build_cache: latent_bytes must be a positive multiple of 16");
        if (!slot_of_entry && n_slots < n)
            return fail(APC_E_ARG, "apc_build_cache: identity slot map needs n_slots >= n");
    } else if (latents || slot_of_entry) {
        return fail(APC_E_ARG, "apc_build_cache: latents/slot_of_entry given with n_slots = 0");
    }

    hipStream_t s = static_cast<hipStream_t>(stream);
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");

    apc_cache* c = new (std::nothrow) apc_cache{};
    if (!c) return fail(APC_E_NOMEM, "apc_build_cache: host allocation failed");
    const int64_t n_pad = apc::factor_pad(n);
    apc::BuildStatus* dst = nullptr;
    apc::BuildStatus hst{};
    if ((e = hipMalloc(&c->fe, sizeof(float) * n_pad)) != hipSuccess) {
        delete c;
        return fail(APC_E_NOMEM, "apc_build_cache: hipMalloc of %lld row factors: %s", (long long)n,
                    hipGetErrorString(e));
    }
    auto cleanup = [&]() {
        if (dst) (void)hipFree(dst);
        (void)hipFree(c->fe);
        delete c;
    };
    if ((e = hipMalloc(&dst, sizeof(apc::BuildStatus))) != hipSuccess) {
        cleanup();
        return fail(APC_E_NOMEM, "apc_build_cache: hipMalloc: %s", hipGetErrorString(e));
    }
    hst.first_bad = ~0ull;
    if ((e = hipMemsetAsync(c->fe + n, 0, sizeof(float) * (n_pad - n), s)) != hipSuccess ||
        (e = hipMemcpyAsync(dst, &hst, sizeof hst, hipMemcpyHostToDevice, s)) != hipSuccess ||
        (e = apc::launch_row_factors(dt, n, d, emb, row_scale, slot_of_entry, n_slots, c->fe, dst, s)) != hipSuccess ||
        (e = hipMemcpyAsync(&hst, dst, sizeof hst, hipMemcpyDeviceToHost, s)) != hipSuccess ||
        (e = hipStreamSynchronize(s)) != hipSuccess) {
        cleanup();
        return hip_fail(e, "apc_build_cache");
    }
    if (hst.flags) {
        const unsigned long long r = hst.first_bad;
        cleanup();
        if (hst.flags & apc::ST_NONFINITE)
            return fail(APC_E_NONFINITE, "apc_build_cache: non-finite values (first bad row %llu)", r);
        if (hst.flags & apc::ST_SCALE)
            return fail(APC_E_NONFINITE, "apc_build_cache: row scale not finite and > 0 (first bad row %llu)", r);
        if (hst.flags & apc::ST_ZERO)
            return fail(APC_E_ZERO_NORM, "apc_build_cache: zero-norm row (first bad row %llu)", r);
        return fail(APC_E_ARG, "apc_build_cache: slot_of_entry out of range (first bad entry %llu)", r);
    }
    (void)hipFree(dst);
    c->dt = dt;
    c->n = n;
    c->d = d;
    c->emb = emb;
    c->row_scale = row_scale;
    c->latents = latents;
    c->n_slots = n_slots;
    c->latent_bytes = latent_bytes;
    c->slot_of_entry = slot_of_entry;
    c->device = dev;
    *out = c;
    return ok();
}

void apc_destroy_cache(apc_cache* c)
{
    if (!c) return;
    (void)hipFree(c->fe);
    delete c;
}

apc_status apc_cache_row_factors(const apc_cache* c, float* out, void* stream)
{
    if (!c || !out) return fail(APC_E_ARG, "apc_cache_row_factors: NULL argument");
    if (apc_status st = check_device("apc_cache_row_factors", c)) return st;
    hipError_t e = hipMemcpyAsync(out, c->fe, sizeof(float) * c->n, hipMemcpyDeviceToDevice,
                                  static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "apc_cache_row_factors");
    return ok();
}

apc_status apc_match_workspace(const apc_cache* c, int32_t b, int32_t k, size_t* bytes)
{
    if (!c || !bytes) return fail(APC_E_ARG, "apc_match_workspace: NULL argument");
    if (b < 0) return fail(APC_E_ARG, "apc_match_workspace: b < 0");
    if (k < 1 || k > APC_MAX_K || k > c->n)
        return fail(APC_E_ARG, "apc_match_workspace: need 1 <= k <= min(n, %d) (k=%d)", APC_MAX_K, k);
    *bytes = b == 0 ? 0 : apc::plan_match(c->dt, c->n, c->d, b, k).bytes;
    return ok();
}

apc_status apc_match_batch(const apc_cache* c, const void* q, const float* q_scale, int32_t b, int32_t k,
                           float* top_score, int32_t* top_idx, void* ws, size_t ws_bytes, void* stream)
{
    if (!c) return fail(APC_E_ARG, "apc_match_batch: NULL cache");
    if (b < 0) return fail(APC_E_ARG, "apc_match_batch: b < 0");
    if (k < 1 || k > APC_MAX_K || k > c->n)
        return fail(APC_E_ARG, "apc_match_batch: need 1 <= k <= min(n, %d) (k=%d)", APC_MAX_K, k);
    if (b == 0) return ok();
    apc_status st = check_rows(c->dt, b, c->d, q, "apc_match_batch queries");
    if (st != APC_OK) return st;
    if ((st = check_device("apc_match_batch", c)) != APC_OK) return st;
    if ((c->dt == APC_E4M3) != (q_scale != nullptr))
        return fail(APC_E_ARG, "apc_match_batch: q_scale is required for e4m3 and only for e4m3");
    if (!top_score || !top_idx || !aligned16(top_score) || !aligned16(top_idx))
        return fail(APC_E_ARG, "apc_match_batch: outputs must be 16-byte aligned device pointers");
    const apc::MatchPlan p = apc::plan_match(c->dt, c->n, c->d, b, k);
    if (!ws || ws_bytes < p.bytes || (reinterpret_cast<uintptr_t>(ws) & 255u))
        return fail(APC_E_WORKSPACE, "apc_match_batch: workspace needs %zu bytes, 256-byte aligned (got %zu)",
                    p.bytes, ws_bytes);
    hipEvent_t ev0 = g_ev_start, ev1 = g_ev_stop;
    g_ev_start = g_ev_stop = nullptr;
    hipError_t e = apc::launch_match(p, c->dt, c->n, c->d, c->emb, c->fe, q, q_scale, b, k, top_score,
                                     top_idx, ws, static_cast<hipStream_t>(stream), ev0, ev1);
    if (e != hipSuccess) return hip_fail(e, "apc_match_batch launch");
    return ok();
}

apc_status apc_match_batch_static(const apc_cache* c, const void* q, const float* q_scale, int32_t b, int32_t k,
                                  float* top_score, int32_t* top_idx, void* stream)
{
    if (!c) return fail(APC_E_ARG, "apc_match_batch_static: NULL cache");
    if (b < 0) return fail(APC_E_ARG, "apc_match_batch_static: b < 0");
    if (k < 1 || k > APC_MAX_K || k > c->n)
        return fail(APC_E_ARG, "apc_match_batch_static: need 1 <= k <= min(n, %d) (k=%d)", APC_MAX_K, k);
    if (b == 0) return ok();
    apc_status st = check_rows(c->dt, b, c->d, q, "apc_match_batch_static queries");
    if (st != APC_OK) return st;
    if ((st = check_device("apc_match_batch_static", c)) != APC_OK) return st;
    if ((c->dt == APC_E4M3) != (q_scale != nullptr))
        return fail(APC_E_ARG, "apc_match_batch_static: q_scale is required for e4m3 and only for e4m3");
    if (!top_score || !top_idx || !aligned16(top_score) || !aligned16(top_idx))
        return fail(APC_E_ARG, "apc_match_batch_static: outputs must be 16-byte aligned device pointers");
    const apc::MatchPlan p = apc::plan_match(c->dt, c->n, c->d, b, k);
    if (p.bytes > (size_t)APC_STATIC_WS_BYTES)
        return fail(APC_E_WORKSPACE,
                    "apc_match_batch_static: b = %d, k = %d needs %zu workspace bytes, more than the %u of the "
                    "static workspace (use apc_match_batch with a workspace of apc_match_workspace() bytes)",
                    b, k, p.bytes, (unsigned)APC_STATIC_WS_BYTES);
    if (c->device < 0 || c->device >= MAX_DEVICES)
        return fail(APC_E_ARG, "apc_match_batch_static: device %d beyond the %d this library tracks", c->device,
                    MAX_DEVICES);
    void* ws = g_scratch_ptr[c->device].load(std::memory_order_acquire);
    if (!ws) {
        // first call on this device (the handle's device is current): the
        // device's own copy of the array
        hipError_t e = hipGetSymbolAddress(&ws, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !ws) return hip_fail(e, "apc_match_batch_static: hipGetSymbolAddress");
        g_scratch_ptr[c->device].store(ws, std::memory_order_release);
    }
    hipEvent_t ev0 = g_ev_start, ev1 = g_ev_stop;
    g_ev_start = g_ev_stop = nullptr;
    hipError_t e = apc::launch_match(p, c->dt, c->n, c->d, c->emb, c->fe, q, q_scale, b, k, top_score, top_idx, ws,
                                     static_cast<hipStream_t>(stream), ev0, ev1);
    if (e != hipSuccess) return hip_fail(e, "apc_match_batch_static launch");
    return ok();
}

namespace {

// Checks the level and instance tables shared by the assignment entry points
// and builds the device table (levels, instances ordered by (level, queue
// desc, index asc), places per level).
// With inst_rand (uniform routing at batch size 1), instances are ordered by
// (level, inst_rand asc, index asc) and each takes at most one query.
apc_status build_assign_table(const char* who, const float* top_score, int32_t ld, int32_t b, int32_t L,
                              const float* theta, const int32_t* K, int32_t n_inst, const int32_t* inst_level,
                              const int32_t* inst_cap, const int32_t* inst_queue, const int32_t* opt_level,
                              const int32_t* out_level, const int32_t* out_inst, const int32_t* out_slot,
                              const int32_t* inst_fill, apc::AssignTable& t, const uint32_t* inst_rand = nullptr)
{
    if (b < 0 || ld < 1) return fail(APC_E_ARG, "%s: need b >= 0 and ld >= 1", who);
    if (L < 0 || L > APC_MAX_LEVELS) return fail(APC_E_TABLE, "%s: need 0 <= L <= %d", who, APC_MAX_LEVELS);
    if (L > 0 && (!theta || !K)) return fail(APC_E_TABLE, "%s: theta/K are NULL", who);
    for (int l = 0; l < L; ++l) {
        if (!std::isfinite(theta[l])) return fail(APC_E_TABLE, "%s: theta[%d] is not finite", who, l);
        if (K[l] <= 0) return fail(APC_E_TABLE, "%s: K[%d] must be > 0", who, l);
        if (l > 0 && !(theta[l] > theta[l - 1]))
            return fail(APC_E_TABLE, "%s: thresholds must be strictly increasing", who);
        if (l > 0 && !(K[l] > K[l - 1])) return fail(APC_E_TABLE, "%s: K must be strictly increasing", who);
    }
    if (n_inst < 0 || n_inst > APC_MAX_INST)
        return fail(APC_E_TABLE, "%s: need 0 <= n_inst <= %d", who, APC_MAX_INST);
    if (n_inst > 0 && (!inst_level || !inst_cap)) return fail(APC_E_TABLE, "%s: instance table is NULL", who);
    int64_t total = 0;
    for (int i = 0; i < n_inst; ++i) {
        if (inst_level[i] < 0 || inst_level[i] > L)
            return fail(APC_E_TABLE, "%s: inst_level[%d] = %d not in 0..%d", who, i, inst_level[i], L);
        if (inst_cap[i] < 0) return fail(APC_E_TABLE, "%s: inst_cap[%d] < 0", who, i);
        total += inst_cap[i];
    }
    if (total > INT32_MAX) return fail(APC_E_TABLE, "%s: total capacity exceeds 2^31 - 1", who);
    if (b > 0 && (!top_score || !opt_level || !out_level || !out_inst || !out_slot))
        return fail(APC_E_ARG, "%s: NULL device buffer", who);
    if (n_inst > 0 && !inst_fill) return fail(APC_E_ARG, "%s: inst_fill is NULL", who);

    t = apc::AssignTable{};
    t.L = L;
    t.n_inst = n_inst;
    for (int l = 0; l < L; ++l) {
        t.theta[l] = theta[l];
        t.K[l + 1] = K[l];
    }
    int order[APC_MAX_INST];
    for (int i = 0; i < n_inst; ++i) order[i] = i;
    std::stable_sort(order, order + n_inst, [&](int a, int c) {
        if (inst_level[a] != inst_level[c]) return inst_level[a] < inst_level[c];
        if (inst_rand) {
            if (inst_rand[a] != inst_rand[c]) return inst_rand[a] < inst_rand[c];
            return a < c;
        }
        const int qa = inst_queue ? inst_queue[a] : 0, qc = inst_queue ? inst_queue[c] : 0;
        if (qa != qc) return qa > qc;
        return a < c;
    });
    auto cap_of = [&](int i) { return inst_rand ? std::min(inst_cap[i], 1) : inst_cap[i]; };
    int j = 0;
    for (int p = 0; p <= L; ++p) {
        t.level_first[p] = j;
        int64_t cum = 0;
        while (j < n_inst && inst_level[order[j]] == p) {
            t.ord_inst[j] = (int16_t)order[j];
            t.ord_cap[j] = cap_of(order[j]);
            t.ord_cum[j] = (int32_t)cum;
            cum += cap_of(order[j]);
            ++j;
        }
        t.level_cap[p] = (int32_t)cum;
    }
    t.level_first[L + 1] = j;
    return APC_OK;
}

}  // namespace

apc_status apc_assign(const float* top_score, int32_t ld, int32_t b, int32_t L, const float* theta,
                      const int32_t* K, int32_t n_inst, const int32_t* inst_level, const int32_t* inst_cap,
                      const int32_t* inst_queue, int32_t* opt_level, int32_t* out_level, int32_t* out_inst,
                      int32_t* out_slot, int32_t* inst_fill, void* stream)
{
    apc::AssignTable t;
    apc_status st = build_assign_table("apc_assign", top_score, ld, b, L, theta, K, n_inst, inst_level, inst_cap,
                                       inst_queue, opt_level, out_level, out_inst, out_slot, inst_fill, t);
    if (st != APC_OK) return st;
    if (b == 0 && n_inst == 0) return ok();
    hipError_t e = apc::launch_assign(t, top_score, ld, b, opt_level, out_level, out_inst, out_slot,
                                      inst_fill, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "apc_assign launch");
    return ok();
}

apc_status apc_assign_load_aware(const float* top_score, int32_t ld, int32_t b, int32_t L, const float* theta,
                                 const int32_t* K, int32_t n_inst, const int32_t* inst_level,
                                 const int32_t* inst_cap, const int32_t* inst_queue, const uint32_t* inst_rand,
                                 int64_t load, int64_t load_threshold, int32_t* routing, int32_t* opt_level,
                                 int32_t* out_level, int32_t* out_inst, int32_t* out_slot, int32_t* inst_fill,
                                 void* stream)
{
    if (!routing) return fail(APC_E_ARG, "apc_assign_load_aware: routing is NULL");
    const bool greedy = load >= load_threshold;
    if (!greedy && n_inst > 0 && !inst_rand)
        return fail(APC_E_ARG, "apc_assign_load_aware: uniform routing needs inst_rand");
    apc::AssignTable t;
    apc_status st = build_assign_table("apc_assign_load_aware", top_score, ld, b, L, theta, K, n_inst, inst_level,
                                       inst_cap, inst_queue, opt_level, out_level, out_inst, out_slot, inst_fill, t,
                                       greedy ? nullptr : inst_rand);
    if (st != APC_OK) return st;
    *routing = greedy ? 1 : 0;
    if (b == 0 && n_inst == 0) return ok();
    hipError_t e = apc::launch_assign(t, top_score, ld, b, opt_level, out_level, out_inst, out_slot, inst_fill,
                                      static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "apc_assign_load_aware launch");
    return ok();
}

apc_status apc_route_plan(int32_t L, const int32_t* K, const int32_t* H, const int32_t* F, int32_t* X,
                          int64_t* degradation)
{
    if (L < 0 || L > APC_MAX_LEVELS) return fail(APC_E_TABLE, "apc_route_plan: need 0 <= L <= %d", APC_MAX_LEVELS);
    if ((L > 0 && !K) || !H || !F || !X) return fail(APC_E_ARG, "apc_route_plan: NULL argument");
    for (int l = 0; l < L; ++l) {
        if (K[l] <= 0) return fail(APC_E_TABLE, "apc_route_plan: K[%d] must be > 0", l);
        if (l > 0 && !(K[l] > K[l - 1])) return fail(APC_E_TABLE, "apc_route_plan: K must be strictly increasing");
    }
    int64_t sh = 0, sf = 0;
    for (int i = 0; i <= L; ++i) {
        if (H[i] < 0 || F[i] < 0) return fail(APC_E_ARG, "apc_route_plan: H[%d] or F[%d] < 0", i, i);
        sh += H[i];
        sf += F[i];
    }
    if (sh > INT32_MAX || sf > INT32_MAX) return fail(APC_E_ARG, "apc_route_plan: sums exceed 2^31 - 1");
    apc::plan_route_host(L, H, F, X);
    if (degradation) {
        int64_t d = 0;
        for (int i = 0; i <= L; ++i)
            for (int j = i + 1; j <= L; ++j)
                d += (int64_t)X[i * (L + 1) + j] * ((int64_t)K[j - 1] - (i > 0 ? K[i - 1] : 0));
        *degradation = d;
    }
    return ok();
}

static apc_status assign_with_plan(const char* who, bool planned, const float* top_score, int32_t ld, int32_t b,
                                   int32_t L, const float* theta, const int32_t* K, int32_t n_inst,
                                   const int32_t* inst_level, const int32_t* inst_cap, const int32_t* inst_queue,
                                   int32_t* plan, int32_t* opt_level, int32_t* out_level, int32_t* out_inst,
                                   int32_t* out_slot, int32_t* inst_fill, void* stream)
{
    apc::AssignTable t;
    apc_status st = build_assign_table(who, top_score, ld, b, L, theta, K, n_inst, inst_level, inst_cap,
                                       inst_queue, opt_level, out_level, out_inst, out_slot, inst_fill, t);
    if (st != APC_OK) return st;
    if (b > APC_MAX_ROUTED_BATCH) return fail(APC_E_ARG, "%s: b = %d exceeds %d", who, b, APC_MAX_ROUTED_BATCH);
    if (!plan) return fail(APC_E_ARG, "%s: plan is NULL", who);
    hipError_t e = apc::launch_assign_plan(t, planned, top_score, ld, b, plan, opt_level, out_level, out_inst,
                                           out_slot, inst_fill, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, who);
    return ok();
}

apc_status apc_assign_routed(const float* top_score, int32_t ld, int32_t b, int32_t L, const float* theta,
                             const int32_t* K, int32_t n_inst, const int32_t* inst_level, const int32_t* inst_cap,
                             const int32_t* inst_queue, const int32_t* plan, int32_t* opt_level,
                             int32_t* out_level, int32_t* out_inst, int32_t* out_slot, int32_t* inst_fill,
                             void* stream)
{
    return assign_with_plan("apc_assign_routed", false, top_score, ld, b, L, theta, K, n_inst, inst_level,
                            inst_cap, inst_queue, const_cast<int32_t*>(plan), opt_level, out_level, out_inst,
                            out_slot, inst_fill, stream);
}

apc_status apc_assign_planned(const float* top_score, int32_t ld, int32_t b, int32_t L, const float* theta,
                              const int32_t* K, int32_t n_inst, const int32_t* inst_level, const int32_t* inst_cap,
                              const int32_t* inst_queue, int32_t* plan, int32_t* opt_level, int32_t* out_level,
                              int32_t* out_inst, int32_t* out_slot, int32_t* inst_fill, void* stream)
{
    return assign_with_plan("apc_assign_planned", true, top_score, ld, b, L, theta, K, n_inst, inst_level,
                            inst_cap, inst_queue, plan, opt_level, out_level, out_inst, out_slot, inst_fill,
                            stream);
}

apc_status apc_resident_best(const apc_cache* c, const float* top_score, const int32_t* top_idx, int32_t ld,
                             int32_t k, int32_t b, float* out_score, int32_t* out_idx, void* stream)
{
    if (!c) return fail(APC_E_ARG, "apc_resident_best: NULL cache");
    if (c->n_slots == 0) return fail(APC_E_ARG, "apc_resident_best: the cache has no latents");
    if (b < 0 || k < 1 || k > APC_MAX_K || ld < k)
        return fail(APC_E_ARG, "apc_resident_best: need b >= 0 and 1 <= k <= min(ld, %d)", APC_MAX_K);
    if (b == 0) return ok();
    if (!top_score || !top_idx || !out_score || !out_idx)
        return fail(APC_E_ARG, "apc_resident_best: NULL device buffer");
    if (apc_status st = check_device("apc_resident_best", c)) return st;
    hipError_t e = apc::launch_resident_best(c->slot_of_entry, c->n, c->n_slots, top_score, top_idx, ld, k, b,
                                             out_score, out_idx, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "apc_resident_best launch");
    return ok();
}

apc_status apc_level_histogram(const int32_t* level, int32_t b, int32_t L, int32_t* hist, void* stream)
{
    if (b < 0 || L < 0 || L > APC_MAX_LEVELS)
        return fail(APC_E_ARG, "apc_level_histogram: need b >= 0 and 0 <= L <= %d", APC_MAX_LEVELS);
    if ((b > 0 && !level) || !hist) return fail(APC_E_ARG, "apc_level_histogram: NULL device buffer");
    hipError_t e = apc::launch_level_histogram(level, b, L, hist, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "apc_level_histogram launch");
    return ok();
}

apc_status apc_merge_shards(const float* scores, const int32_t* idx, int32_t g, int32_t b, int32_t k_in,
                            const int32_t* offsets, int32_t k, float* out_score, int32_t* out_idx, void* stream)
{
    if (g < 1 || g > APC_MAX_SHARDS || b < 0 || k < 1 || k > APC_MAX_K || k_in < 1 || k_in > APC_MAX_K)
        return fail(APC_E_ARG, "apc_merge_shards: need 1 <= g <= %d, b >= 0, 1 <= k, k_in <= %d", APC_MAX_SHARDS,
                    APC_MAX_K);
    if (!offsets) return fail(APC_E_ARG, "apc_merge_shards: offsets is NULL");
    apc::ShardOffsets off{};
    for (int s = 0; s < g; ++s) {
        if (offsets[s] < 0) return fail(APC_E_ARG, "apc_merge_shards: offsets[%d] < 0", s);
        off.v[s] = offsets[s];
    }
    if (b == 0) return ok();
    if (!scores || !idx || !out_score || !out_idx) return fail(APC_E_ARG, "apc_merge_shards: NULL device buffer");
    hipError_t e = apc::launch_merge_shards(scores, idx, g, b, k_in, off, k, out_score, out_idx,
                                            static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "apc_merge_shards launch");
    return ok();
}

static apc_status gather_impl(const char* who, const apc_cache* c, const int32_t* top_idx, int32_t ld, int32_t b,
                              const int32_t* out_level, const int32_t* out_inst, const int32_t* out_slot,
                              int32_t n_inst, int32_t slots_per_inst, int32_t lps, void* batch_latents,
                              int32_t* hit, void* stream)
{
    if (!c) return fail(APC_E_ARG, "%s: NULL cache", who);
    if (c->n_slots == 0) return fail(APC_E_ARG, "%s: the cache has no latents", who);
    if (b < 0 || ld < 1 || n_inst < 0 || slots_per_inst < 0)
        return fail(APC_E_ARG, "%s: need b >= 0, ld >= 1, n_inst >= 0, slots_per_inst >= 0", who);
    if (lps < 1 || lps > APC_MAX_LEVELS || c->n_slots % lps != 0)
        return fail(APC_E_ARG, "%s: levels_per_slot must be in 1..%d and divide the cache's %lld latents", who,
                    APC_MAX_LEVELS, (long long)c->n_slots);
    if (b == 0) return ok();
    if (!top_idx || !out_level || !out_inst || !out_slot || !hit)
        return fail(APC_E_ARG, "%s: NULL device buffer", who);
    if ((int64_t)n_inst * slots_per_inst > 0 && (!batch_latents || !aligned16(batch_latents)))
        return fail(APC_E_ARG, "%s: batch_latents must be 16-byte aligned", who);
    if (apc_status st = check_device(who, c)) return st;
    hipError_t e = apc::launch_gather(c->latents, c->n, c->n_slots, c->latent_bytes, c->slot_of_entry,
                                      top_idx, ld, b, out_level, out_inst, out_slot, n_inst, slots_per_inst, lps,
                                      batch_latents, hit, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, who);
    return ok();
}

apc_status apc_gather_latents(const apc_cache* c, const int32_t* top_idx, int32_t ld, int32_t b,
                              const int32_t* out_level, const int32_t* out_inst, const int32_t* out_slot,
                              int32_t n_inst, int32_t slots_per_inst, void* batch_latents, int32_t* hit,
                              void* stream)
{
    return gather_impl("apc_gather_latents", c, top_idx, ld, b, out_level, out_inst, out_slot, n_inst,
                       slots_per_inst, 1, batch_latents, hit, stream);
}

apc_status apc_gather_latents_at_level(const apc_cache* c, const int32_t* top_idx, int32_t ld, int32_t b,
                                       const int32_t* out_level, const int32_t* out_inst, const int32_t* out_slot,
                                       int32_t n_inst, int32_t slots_per_inst, int32_t levels_per_slot,
                                       void* batch_latents, int32_t* hit, void* stream)
{
    return gather_impl("apc_gather_latents_at_level", c, top_idx, ld, b, out_level, out_inst, out_slot, n_inst,
                       slots_per_inst, levels_per_slot, batch_latents, hit, stream);
}

}  // extern "C"
