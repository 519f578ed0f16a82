/*
 * Reference implementation of the prompt -> cached-state matching step.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may link or call
 * this file: only the tests, the smoke check and the CPU-baseline leg of the
 * benchmark use it.  It shares no code, header, table or constant with the
 * HIP library.
 *
 * It follows the paper's Approach section: the Query Dispatcher's Optimal-K
 * Selector "retrieves the nearest cache and determines the optimal K"; the
 * optimal K is the largest skip that keeps quality; prompts that cannot be
 * placed at their optimal K are redirected either to a slower model (K' < K)
 * or to the closest faster one (K' > K) (Resource Controller paragraph and
 * Eq. 1, which charges degradation only for K' > K); and greedy routing
 * fills the worker with the longest queue first (route-and-batch paragraph).
 * The paper gives no formulas for these steps; the readings taken here are:
 *
 *   score   s(q,e) = clamp(<q,e> / sqrt(|q|^2 |e|^2), -1, 1), cosine of the
 *           stored vectors, exact brute force over all entries, in float64
 *           (one square root of the product of the squared norms, so that a
 *           cosine that is a simple fraction comes out exactly);
 *   top-k   the first k entries in the order (score desc, index asc);
 *   level   lambda = #{l in 1..L : best >= theta_l}, best = top-1 score,
 *           theta given as float32 (level 0 = no skip);
 *   assign  rounds r = 0..L over preference lists
 *           [lambda, lambda-1, .., 0, lambda+1, .., L]; in each round the
 *           unassigned queries, in index order, take a place at their r-th
 *           preference while that level has capacity left;
 *   slot    within a level, admissions in order fill the instances ordered
 *           by (queue length desc, index asc), each up to its capacity;
 *   gather  an assigned query at a level > 0 whose top-1 entry has a
 *           resident latent gets that latent copied to its (instance, slot).
 *
 * Plain loops, no blocking: decoding is exact (f16/bf16/e4m3fn widen exactly
 * to float64; the e4m3fn value times its float32 row scale is exact too).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

enum { OR_F32 = 0, OR_F16 = 1, OR_BF16 = 2, OR_E4M3 = 3 };
enum { OR_OK = 0, OR_E_ARG = 1, OR_E_NONFINITE = 2, OR_E_ZERO_NORM = 3, OR_E_NOMEM = 4 };

/* ---- decoding of the stored formats (IEEE binary16, bfloat16, OCP e4m3fn) ---- */

static double dec_f16(uint16_t h)
{
    int sign = h >> 15, ex = (h >> 10) & 31, man = h & 1023;
    double v;
    if (ex == 0)
        v = ldexp((double)man, -24);                 /* subnormal: man * 2^-24 */
    else if (ex == 31)
        v = man ? NAN : INFINITY;
    else
        v = ldexp((double)(1024 + man), ex - 25);    /* (1 + man/1024) * 2^(ex-15) */
    return sign ? -v : v;
}

static double dec_bf16(uint16_t h)
{
    uint32_t bits = (uint32_t)h << 16;               /* upper half of a binary32 */
    float f;
    memcpy(&f, &bits, 4);
    return (double)f;
}

static double dec_e4m3(uint8_t c)
{
    int sign = c >> 7, ex = (c >> 3) & 15, man = c & 7;
    double v;
    if (ex == 15 && man == 7)
        return NAN;                                  /* the only NaN codes: 0x7F, 0xFF */
    if (ex == 0)
        v = ldexp((double)man, -9);                  /* subnormal: man/8 * 2^(1-7) */
    else
        v = ldexp((double)(8 + man), ex - 10);       /* (1 + man/8) * 2^(ex-7) */
    return sign ? -v : v;
}

static size_t elem_bytes(int dt)
{
    switch (dt) {
    case OR_F32: return 4;
    case OR_F16: case OR_BF16: return 2;
    case OR_E4M3: return 1;
    default: return 0;
    }
}

/* decoded value of every 16-bit and 8-bit code, filled once from the
   functions above (a memo of them, nothing more) */
static double lut_f16[65536], lut_bf16[65536], lut_e4m3[256];
static int lut_ready = 0;

__attribute__((constructor)) static void fill_luts(void)
{
    for (int c = 0; c < 65536; ++c) {
        lut_f16[c] = dec_f16((uint16_t)c);
        lut_bf16[c] = dec_bf16((uint16_t)c);
    }
    for (int c = 0; c < 256; ++c) lut_e4m3[c] = dec_e4m3((uint8_t)c);
    lut_ready = 1;
}

/* value of element i of row r, scaled by the row's float32 scale for e4m3 */
static inline double elem(int dt, const void* base, const float* scale, int64_t r, int32_t d, int32_t i)
{
    int64_t off = r * (int64_t)d + i;
    switch (dt) {
    case OR_F32: return (double)((const float*)base)[off];
    case OR_F16: return lut_f16[((const uint16_t*)base)[off]];
    case OR_BF16: return lut_bf16[((const uint16_t*)base)[off]];
    default: return lut_e4m3[((const uint8_t*)base)[off]] * (double)scale[r];
    }
}

int oracle_decode(int dt, const void* rows, const float* scale, int64_t n, int32_t d, double* out)
{
    if (!elem_bytes(dt) || n < 0 || d < 1 || (dt == OR_E4M3 && !scale)) return OR_E_ARG;
    for (int64_t r = 0; r < n; ++r)
        for (int32_t i = 0; i < d; ++i)
            out[r * d + i] = elem(dt, rows, scale, r, d, i);
    return OR_OK;
}

/* Squared Euclidean norm of each row (sequential sum of squares; rows run in
 * parallel).  Returns the first bad row's status: a non-finite element makes
 * the sum non-finite (OR_E_NONFINITE); an all-zero row gives 0 (OR_E_ZERO_NORM). */
int oracle_row_sqnorms(int dt, const void* rows, const float* scale, int64_t n, int32_t d,
                       double* sq, int64_t* bad_row)
{
    if (!elem_bytes(dt) || n < 0 || d < 1 || (dt == OR_E4M3 && !scale) || !lut_ready) return OR_E_ARG;
#ifdef _OPENMP
#pragma omp parallel for schedule(static)
#endif
    for (int64_t r = 0; r < n; ++r) {
        double ss = 0.0;
        for (int32_t i = 0; i < d; ++i) {
            double x = elem(dt, rows, scale, r, d, i);
            ss += x * x;
        }
        sq[r] = ss;
    }
    *bad_row = -1;
    for (int64_t r = 0; r < n; ++r) {
        if (!isfinite(sq[r])) { *bad_row = r; return OR_E_NONFINITE; }
        if (!(sq[r] > 0.0)) { *bad_row = r; return OR_E_ZERO_NORM; }
    }
    return OR_OK;
}

/* cosine of a decoded query row qv (squared norm sq_q) and stored entry row ei
   (squared norm sq_e), clamped to [-1, 1] */
static double score(int dt, const double* qv, double sq_q,
                    const void* e, const float* es, int64_t ei, double sq_e, int32_t d)
{
    double dot = 0.0;
    for (int32_t i = 0; i < d; ++i)
        dot += qv[i] * elem(dt, e, es, ei, d, i);
    double s = dot / sqrt(sq_q * sq_e);
    if (s > 1.0) s = 1.0;
    if (s < -1.0) s = -1.0;
    return s;
}

/* a precedes b in the order (score desc, index asc) */
static int before(double sa, int64_t ia, double sb, int64_t ib)
{
    return sa > sb || (sa == sb && ia < ib);
}

/*
 * Scores of given (query row, entry row) pairs.
 */
int oracle_pair_scores(int dt, const void* q, const float* qs, const double* q_sq,
                       const void* e, const float* es, const double* e_sq, int32_t d,
                       int64_t npairs, const int64_t* qi, const int64_t* ei, double* out)
{
    if (!elem_bytes(dt) || d < 1 || !lut_ready) return OR_E_ARG;
    double* qv = malloc(sizeof(double) * (size_t)d);
    if (!qv) return OR_E_NOMEM;
    for (int64_t p = 0; p < npairs; ++p) {
        for (int32_t i = 0; i < d; ++i) qv[i] = elem(dt, q, qs, qi[p], d, i);
        out[p] = score(dt, qv, q_sq[qi[p]], e, es, ei[p], e_sq[ei[p]], d);
    }
    free(qv);
    return OR_OK;
}

/*
 * Exact top-k of every query row against all n entry rows: for each query the
 * k entries that come first in the order (score desc, index asc).  Squared
 * norms are passed in (from oracle_row_sqnorms).  Queries are independent; OpenMP runs
 * them on `threads` threads (0 = runtime default).
 */
int oracle_topk(int dt, const void* q, const float* qs, const double* q_sq, int64_t b,
                const void* e, const float* es, const double* e_sq, int64_t n,
                int32_t d, int32_t k, int threads, double* top_s, int64_t* top_i)
{
    if (!elem_bytes(dt) || d < 1 || k < 1 || k > n || b < 0 || !lut_ready) return OR_E_ARG;
    int failed = 0;
#ifdef _OPENMP
    if (threads > 0) omp_set_num_threads(threads);
#pragma omp parallel for schedule(dynamic, 1)
#endif
    for (int64_t qi = 0; qi < b; ++qi) {
        double* ls = top_s + qi * k;
        int64_t* li = top_i + qi * k;
        double* qv = malloc(sizeof(double) * (size_t)d);
        if (!qv) { failed = 1; continue; }
        for (int32_t i = 0; i < d; ++i) qv[i] = elem(dt, q, qs, qi, d, i);
        int32_t filled = 0;
        for (int64_t ei = 0; ei < n; ++ei) {
            double s = score(dt, qv, q_sq[qi], e, es, ei, e_sq[ei], d);
            if (filled == k && !before(s, ei, ls[k - 1], li[k - 1]))
                continue;
            /* insert into the sorted list, dropping the last one if full */
            int32_t p = filled < k ? filled++ : k - 1;
            while (p > 0 && before(s, ei, ls[p - 1], li[p - 1])) {
                ls[p] = ls[p - 1];
                li[p] = li[p - 1];
                --p;
            }
            ls[p] = s;
            li[p] = ei;
        }
        free(qv);
    }
    return failed ? OR_E_NOMEM : OR_OK;
}

/* level of each query: number of thresholds (float32, strictly increasing) at or below its best score */
int oracle_levels(const double* best, int64_t b, int32_t L, const float* theta, int32_t* level)
{
    if (b < 0 || L < 0) return OR_E_ARG;
    for (int32_t l = 1; l < L; ++l)
        if (!(theta[l] > theta[l - 1])) return OR_E_ARG;
    for (int64_t q = 0; q < b; ++q) {
        int32_t lv = 0;
        for (int32_t l = 0; l < L; ++l)
            if (best[q] >= (double)theta[l]) ++lv;
        level[q] = lv;
    }
    return OR_OK;
}

/* r-th entry of the preference list [lam, lam-1, .., 0, lam+1, .., L] */
static int32_t pref(int32_t lam, int32_t r)
{
    return r <= lam ? lam - r : r;
}

/*
 * Capacity-constrained assignment of queries (given their levels) to
 * instances.  Outputs per query: assigned level, instance and slot (-1 when
 * no capacity was left anywhere); per instance: number of queries placed.
 */
int oracle_assign(const int32_t* level, int64_t b, int32_t L, int32_t n_inst,
                  const int32_t* inst_level, const int32_t* inst_cap, const int32_t* inst_queue,
                  int32_t* out_level, int32_t* out_inst, int32_t* out_slot, int32_t* inst_fill)
{
    if (b < 0 || L < 0 || n_inst < 0) return OR_E_ARG;
    for (int64_t q = 0; q < b; ++q)
        if (level[q] < 0 || level[q] > L) return OR_E_ARG;
    for (int32_t i = 0; i < n_inst; ++i)
        if (inst_level[i] < 0 || inst_level[i] > L || inst_cap[i] < 0) return OR_E_ARG;

    int64_t* R = calloc((size_t)L + 1, sizeof(int64_t));      /* capacity per level */
    int64_t* used = calloc((size_t)L + 1, sizeof(int64_t));
    int64_t* rank = malloc(sizeof(int64_t) * (size_t)(b ? b : 1));
    if (!R || !used || !rank) { free(R); free(used); free(rank); return OR_E_NOMEM; }
    for (int32_t i = 0; i < n_inst; ++i) R[inst_level[i]] += inst_cap[i];

    for (int64_t q = 0; q < b; ++q) out_level[q] = -1;
    for (int32_t r = 0; r <= L; ++r)
        for (int64_t q = 0; q < b; ++q) {
            if (out_level[q] >= 0) continue;
            int32_t p = pref(level[q], r);
            if (used[p] < R[p]) {
                out_level[q] = p;
                rank[q] = used[p]++;
            }
        }

    /* all instances sorted by (level asc, queue desc, index asc): insertion sort */
    int32_t* order = malloc(sizeof(int32_t) * (size_t)(n_inst ? n_inst : 1));
    if (!order) { free(R); free(used); free(rank); return OR_E_NOMEM; }
    for (int32_t i = 0; i < n_inst; ++i) {
        int32_t j = i;
        while (j > 0) {
            int32_t a = order[j - 1];
            int32_t qa = inst_queue ? inst_queue[a] : 0, qi = inst_queue ? inst_queue[i] : 0;
            int after = inst_level[a] > inst_level[i] ||
                        (inst_level[a] == inst_level[i] && (qa < qi || (qa == qi && a > i)));
            if (!after) break;
            order[j] = a;
            --j;
        }
        order[j] = i;
    }

    /* the admission of rank t at level lam goes to the level's instance whose
       cumulative capacity (in the order above) first exceeds t */
    for (int32_t i = 0; i < n_inst; ++i) inst_fill[i] = 0;
    for (int64_t q = 0; q < b; ++q) {
        out_inst[q] = out_slot[q] = -1;
        if (out_level[q] < 0) continue;
        int64_t t = rank[q];
        for (int32_t j = 0; j < n_inst; ++j) {
            int32_t i = order[j];
            if (inst_level[i] != out_level[q]) continue;
            if (t < inst_cap[i]) {
                out_inst[q] = i;
                out_slot[q] = (int32_t)t;
                inst_fill[i] += 1;
                break;
            }
            t -= inst_cap[i];
        }
    }
    free(order);
    free(R); free(used); free(rank);
    return OR_OK;
}

/*
 * Latent gather: for every assigned query at a level > 0 whose top-1 entry
 * has a resident latent, copy that latent to batch[inst][slot].  slot_of_entry
 * may be NULL (entry i lives in slot i).  hit[q] = 1 when copied.
 */
int oracle_gather(const int64_t* top1, int64_t b, const int32_t* out_level, const int32_t* out_inst,
                  const int32_t* out_slot, const int32_t* slot_of_entry, int64_t n_entries,
                  const uint8_t* pool, int64_t n_slots, int64_t latent_bytes,
                  int32_t n_inst, int32_t slots_per_inst, uint8_t* batch, int32_t* hit)
{
    if (b < 0 || latent_bytes < 0) return OR_E_ARG;
    for (int64_t q = 0; q < b; ++q) {
        hit[q] = 0;
        if (out_level[q] <= 0 || top1[q] < 0 || top1[q] >= n_entries) continue;
        int64_t slot = slot_of_entry ? slot_of_entry[top1[q]] : top1[q];
        if (slot < 0 || slot >= n_slots) continue;
        if (out_inst[q] < 0 || out_inst[q] >= n_inst || out_slot[q] < 0 || out_slot[q] >= slots_per_inst)
            return OR_E_ARG;
        memcpy(batch + ((int64_t)out_inst[q] * slots_per_inst + out_slot[q]) * latent_bytes,
               pool + slot * latent_bytes, (size_t)latent_bytes);
        hit[q] = 1;
    }
    return OR_OK;
}

int oracle_max_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}
